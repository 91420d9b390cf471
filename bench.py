"""Benchmark of the masked convolution backward pass (dX + dW) on one MI355X.

    python bench.py [--gpus 1] [--steps 50] [--warmup 200] [--no-cpu]

Workload: the VGG-style 3x3 layer N=32, C=K=256, 56x56, stride 1, pad 1,
bf16 inputs with fp32 accumulation; X = relu(N(0,1) - 0.25) (footprint
density 0.401), dY = N(0,1) * Bernoulli(0.4), He-initialised W; seeded
synthetic data.  Inputs (X, W, dY and the two packed footprints) are resident
in device memory before timing starts.

One step is the whole sparse backward of the layer, one conv_bwd_sparse call
on one stream: the preparation launch (filter transform, compaction counts of
the X footprint, dY block occupancy), the skipping weight-gradient GEMM, the
masked data-gradient GEMM (whose tail workgroups sum the weight gradient's
split-K partials) and the data gradient's split reduction.  The dense
comparison step is the same call with no footprints and CBW_FLAG_NO_SKIP.
The same work through the three separate entry points (conv_bwd_data_masked,
conv_bwd_weight_sparse) is timed beside it.
Footprint packing (cbw_relu_mask_pack, cbw_nonzero_mask_pack) belongs to the
forward pass and is timed separately.

Timing: after the warm-up, sparse and dense steps are timed in --rounds
alternating rounds (the order flips every round) of exactly --steps steps,
each round between synchronizations; step times are the medians over rounds.

Prints one JSON line.  value = dense-equivalent TFLOP/s of the sparse step,
(F_conv(dX) + F_conv(dW)) / t, with F_conv = 2 N K P Q C R S per gradient;
useful TFLOP/s counts only live outputs of dX (2 nnz(mask) K R S) and non-zero
entries of dY for dW (2 nnz(dY) C R S).  roofline.frac is the dominant GEMM
kernel's useful FLOPs over its duration against the 2.5 PFLOP/s bf16 peak
(also against the measured peak, and the executed-FLOP rate beside it).  The
same run checks the timed step's outputs against the oracle on sampled
coordinates (exit status 1 on a mismatch) and times the VGG-16 stack.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-context", action="store_true",
                    help="skip the context timings through torch (MIOpen convolution, hipBLASLt GEMMs)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="CPU baseline time budget")
    ap.add_argument("--sweep", choices=["config4", "config3", "config5", "config5_pooled", "elementwise"], default=None,
                    help="instead of the main line, time the sparse and dense steps over a workload set "
                         "(one JSON line per layer or density point)")
    ap.add_argument("--rounds", type=int, default=5,
                    help="alternating sparse/dense timing rounds of --steps steps each (medians reported)")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured-peak microbenchmarks")
    ap.add_argument("--no-stack", action="store_true", help="skip the VGG-16 stack timing")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 256 MiB device copy three times (reference for HBM byte counters)")
    ap.add_argument("--trace-layer", default=None, metavar="NAME",
                    help="instead of the main line, run one named layer's combined sparse and dense steps in "
                         "alternating rounds of --steps steps (after --warmup of each), a small fill kernel "
                         "marking every round, for rocprofv3 kernel traces and counter passes; prints the "
                         "round order and per-round times as JSON")
    return ap.parse_args()


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


_HIP = None


def _hip():
    global _HIP
    if _HIP is None:
        import ctypes
        _HIP = ctypes.CDLL("libamdhip64.so")
    return _HIP


def _fence_free_event():
    """A raw timing hipEvent_t created with hipEventDisableSystemFence."""
    import ctypes
    ev = ctypes.c_void_p()
    if _hip().hipEventCreateWithFlags(ctypes.byref(ev), 0x20000000) != 0:
        raise RuntimeError("hipEventCreateWithFlags failed")
    return ev.value


def _event_ms(a, b):
    import ctypes
    ms = ctypes.c_float()
    if _hip().hipEventSynchronize(ctypes.c_void_p(b)) != 0 or \
            _hip().hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
        raise RuntimeError("hipEventElapsedTime failed")
    return ms.value


def _event_destroy(e):
    import ctypes
    _hip().hipEventDestroy(ctypes.c_void_p(e))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build targets a single MI355X (data-parallel "
              "sharding over the batch is described in DESIGN.md, not run). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.sweep:
        run_sweep(args)
        return
    if args.trace_layer:
        trace_layer(args)
        return

    import numpy as np
    import torch

    import paper_2109_07710_amd as cb
    import workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    spec = wl.config2()[0]
    log("drawing workload %s" % spec.name)
    t_cpu = wl.draw(spec)
    x, w, dy = (t_cpu[k].to(dev) for k in ("x", "w", "dy"))
    desc = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad)
    stream = torch.cuda.current_stream()

    xm = torch.empty(cb.cbw_mask_words(desc), dtype=torch.int32, device=dev)
    dym = torch.empty(cb.cbw_dy_mask_words(desc), dtype=torch.int32, device=dev)
    dx = torch.empty_like(x)
    dw = torch.empty((spec.K, spec.R, spec.S, spec.C), dtype=torch.float32, device=dev)
    ws_m = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED, dev)
    ws_d = cb.workspace(desc, cb.CBW_OP_BWD_DATA, dev)
    ws_w = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT, dev)

    def pack():
        cb.cbw_relu_mask_pack(desc, x, xm)
        cb.cbw_nonzero_mask_pack(desc.dtype, dy.numel(), dy, dym)

    ws_b = cb.workspace(desc, cb.CBW_OP_BWD_BOTH, dev)

    def sparse_dx():
        cb.conv_bwd_data_masked(desc, dy, w, xm, dx, ws_m, 0)

    def sparse_dw():
        cb.conv_bwd_weight_sparse(desc, x, dy, dym, dw, ws_w, 0)

    def dense_dx():
        cb.conv_bwd_data(desc, dy, w, dx, ws_d)

    def dense_dw():
        cb.conv_bwd_weight_sparse(desc, x, dy, None, dw, ws_w, cb.CBW_FLAG_NO_SKIP)

    # The step is one conv_bwd_sparse call: both gradients, with the integer
    # passes of both in one launch, the weight-gradient GEMM, and the
    # data-gradient GEMM whose tail workgroups sum the weight gradient's
    # split-K partials; the skipping step adds the data gradient's split
    # reduction (gather mode decides its split on the device), four launches
    # against the dense step's three.  The dense step is the same call with
    # no footprint and CBW_FLAG_NO_SKIP.  (Forking
    # the two gradients onto two streams was measured slower: both GEMMs want
    # every CU.)
    def sparse_step():
        cb.conv_bwd_sparse(desc, x, dy, w, xm, dym, dx, dw, ws_b, 0)

    def dense_step():
        cb.conv_bwd_sparse(desc, x, dy, w, None, None, dx, dw, ws_b, cb.CBW_FLAG_NO_SKIP)

    # The same work through the separate calls (three entry points).
    def separate_sparse_step():
        sparse_dx()
        sparse_dw()

    def separate_dense_step():
        dense_dx()
        dense_dw()

    def timed(fn, steps, per_kernel=False):
        """Mean ms per call of fn over `steps` back-to-back calls, HIP events
        on the launch stream, synchronized on both sides; optionally the mean
        duration of the data- and weight-gradient GEMM kernels from events the
        library records around their dispatch.  Those per-kernel events are
        created without the system-scope fence (hipEventDisableSystemFence):
        default timing events write back and invalidate the caches when they
        are recorded, which slows the kernel they bracket."""
        evs = []
        if per_kernel:
            for _ in range(steps):
                evs.append([_fence_free_event() for _ in range(4)])
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for i in range(steps):
            if per_kernel:
                cb.cbw_set_profile_events(cb.CBW_OP_BWD_DATA, evs[i][0], evs[i][1])
                cb.cbw_set_profile_events(cb.CBW_OP_BWD_WEIGHT, evs[i][2], evs[i][3])
            fn()
        t1.record(stream)
        torch.cuda.synchronize()
        if per_kernel:
            cb.cbw_set_profile_events(cb.CBW_OP_BWD_DATA)
            cb.cbw_set_profile_events(cb.CBW_OP_BWD_WEIGHT)
        ms = t0.elapsed_time(t1) / steps
        kern = None
        if per_kernel:
            kern = (float(np.mean([_event_ms(p[0], p[1]) for p in evs])),
                    float(np.mean([_event_ms(p[2], p[3]) for p in evs])))
            for p in evs:
                for e in p:
                    _event_destroy(e)
        return ms, kern

    # footprints (forward-pass side, timed separately)
    pack()
    torch.cuda.synchronize()
    ms_pack, _ = timed(pack, 10)

    log("warmup %d" % args.warmup)
    for _ in range(args.warmup):
        sparse_step()
        dense_step()
    torch.cuda.synchronize()

    # Sparse and dense steps timed in alternating rounds (the order flips
    # every round), each round exactly `steps` steps between synchronizations;
    # the medians over rounds are the step times, so clock ramp-up after a
    # short warm-up biases neither side.
    log("timing %d rounds of %d sparse and %d dense steps" % (args.rounds, args.steps, args.steps))
    per_round = alternate({"sparse": sparse_step, "dense": dense_step}, lambda fn: timed(fn, args.steps)[0],
                          args.rounds)
    ms_sparse = float(np.median(per_round["sparse"]))
    ms_dense = float(np.median(per_round["dense"]))
    log("timing %d sparse steps with per-kernel events" % args.steps)
    ms_sparse_k, (ms_dx_gemm, ms_dw_gemm) = timed(sparse_step, args.steps, per_kernel=True)
    _, (ms_dx_gemm_dense, ms_dw_gemm_dense) = timed(dense_step, args.steps, per_kernel=True)

    sparse_step()
    torch.cuda.synchronize()
    st_dx = st_dw = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_BOTH, ws_b)
    log("parity of the timed step's outputs against the oracle (sampled)")
    parity = check_against_oracle(spec, t_cpu, dx, dw, x)

    nnz_mask = int(torch.count_nonzero(x > 0).item())
    nnz_dy = int(torch.count_nonzero(dy).item())
    f_conv = spec.dense_flops()                          # per gradient
    f_useful_dx = 2 * nnz_mask * spec.K * spec.R * spec.S
    f_useful_dw = 2 * nnz_dy * spec.C * spec.R * spec.S
    dense_eq = 2 * f_conv / (ms_sparse * 1e-3) / 1e12
    useful = (f_useful_dx + f_useful_dw) / (ms_sparse * 1e-3) / 1e12
    exec_frac_dx = st_dx.rows_live / st_dx.rows_total
    exec_frac_dw = 1.0 - st_dw.blocks_skipped / max(st_dw.blocks_total, 1)
    f_exec = f_conv * exec_frac_dx + f_conv * exec_frac_dw

    peaks = None
    if not args.no_peaks:
        log("measured peaks (matrix-core loop, HBM streams)")
        peaks = measure_peaks(torch, stream)

    # Dominant kernel: the weight-gradient GEMM, the longer of the two pure
    # GEMM launches (the data-gradient launch of the combined call also sums
    # the weight gradient's split-K partials in its tail workgroups, so its
    # duration is not a GEMM's alone; it is reported as dx_launch_ms).
    # `achieved` counts the useful FLOPs of its gradient (non-zero dY
    # entries), the figure the target is stated in; the executed
    # (dense-equivalent over the blocks actually run) rate is reported
    # beside it.
    tiling = cb.cbw_data_tiling(desc)   # all pixels are live here, so the gather mode tiles alike
    kern = {"dx_gemm": ms_dx_gemm, "dw_gemm": ms_dw_gemm}
    dom = "dw_gemm"
    dom_useful = f_useful_dx if dom == "dx_gemm" else f_useful_dw
    dom_exec = f_conv * (exec_frac_dx if dom == "dx_gemm" else exec_frac_dw)
    achieved = dom_useful / (kern[dom] * 1e-3) / 1e12
    achieved_exec = dom_exec / (kern[dom] * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic_for(dom),
                "flops": "useful: %s" % ("2 nnz(mask) K R S (live dX outputs)" if dom == "dx_gemm"
                                         else "2 nnz(dY) C R S (non-zero dY entries)"),
                "kernel": {"dx_gemm": "bwd_data_kernel<unsigned short, 2, true, 0> (bf16, gather, %d-channel x %d-pixel "
                                      "tiles of %d-row capacity)" % (tiling[0], tiling[2], tiling[1]),
                           "dw_gemm": "bwd_weight_tr_kernel<256> (bf16, 256-wide output-channel tile)"}[dom],
                "kernel_ms": round(kern[dom], 4), "flops_per_launch": dom_useful,
                "executed": {"achieved": round(achieved_exec, 2),
                             "frac": round(achieved_exec / PEAK_BF16_TFLOPS, 4), "flops_per_launch": dom_exec},
                "step_useful_frac": round(useful / PEAK_BF16_TFLOPS, 4),
                "step_dense_equiv_frac": round(dense_eq / PEAK_BF16_TFLOPS, 4)}
    if peaks and "mfma_bf16_tflops" in peaks:
        pk = peaks["mfma_bf16_tflops"]
        roofline["measured_peak"] = {"tflops": pk, "frac": round(achieved / pk, 4),
                                     "frac_executed": round(achieved_exec / pk, 4),
                                     "step_useful_frac": round(useful / pk, 4)}

    # The forward convolution with the ReLU and the footprint fused (the
    # producer of this layer's footprint), timed as a whole call on the same layer.
    log("timing %d forward calls" % args.steps)
    y_fwd = torch.empty((spec.N, desc.P, desc.Q, spec.K), dtype=x.dtype, device=dev)
    ym_fwd = torch.empty(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device=dev)
    ws_f = cb.workspace(desc, cb.CBW_OP_FWD, dev)

    def fwd():
        cb.conv_fwd_relu_mask(desc, x, w, y_fwd, ym_fwd, ws_f)

    for _ in range(max(args.warmup // 4, 5)):
        fwd()
    ms_fwd, _ = timed(fwd, args.steps)
    del y_fwd, ym_fwd, ws_f

    # Per-step distribution of both steps, hot (operands left in the caches by
    # the step before) and cold (the 256 MB last-level cache flushed by
    # writing 512 MB before every step), each step bracketed by its own
    # events; sparse and dense steps interleaved.
    log("per-step distribution, hot and cold")
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)

    def distribution(cold, n=max(10, min(args.steps, 40))):
        per = {"sparse": [], "dense": []}
        for i in range(n):
            for name, fn in (("sparse", sparse_step), ("dense", dense_step))[::(1 if i % 2 == 0 else -1)]:
                if cold:
                    flush.fill_(i & 0xFF)
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                fn()
                b.record(stream)
                torch.cuda.synchronize()
                per[name].append(a.elapsed_time(b))
        out = {}
        for name, v in per.items():
            q = np.percentile(v, [10, 50, 90])
            out[name] = {"p10_ms": round(float(q[0]), 4), "median_ms": round(float(q[1]), 4),
                         "p90_ms": round(float(q[2]), 4)}
        out["speedup_median"] = round(out["dense"]["median_ms"] / out["sparse"]["median_ms"], 4)
        out["steps"] = n
        return out

    dist = {"hot": distribution(False), "cold": distribution(True)}
    del flush

    # The semantic equivalent without output sparsity: the dense step followed
    # by a separate multiply of dX with the 0/1 ReLU derivative.
    relu_d = (x > 0).to(x.dtype)

    def dense_mask_step():
        dense_dx()
        dx.mul_(relu_d)
        dense_dw()

    for _ in range(10):
        separate_sparse_step()
        separate_dense_step()
        dense_mask_step()
    extra = alternate({"separate_sparse": separate_sparse_step, "separate_dense": separate_dense_step,
                       "dense_mask": dense_mask_step, "dense": dense_step},
                      lambda fn: timed(fn, args.steps)[0], 3)
    ms_sep_sparse = float(np.median(extra["separate_sparse"]))
    ms_sep_dense = float(np.median(extra["separate_dense"]))
    ms_dense_mask = float(np.median(extra["dense_mask"]))
    ms_dense_here = float(np.median(extra["dense"]))
    del relu_d

    # NCHW callers: the same step through the library's boundary transposes
    # (activations and footprints in NCHW order), timed apart from the path.
    log("timing %d sparse steps with NCHW tensors" % args.steps)
    desc_n = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad,
                              act_layout="nchw")
    x_n = x.permute(0, 3, 1, 2).contiguous()
    dy_n = dy.permute(0, 3, 1, 2).contiguous()
    dx_n = torch.empty_like(x_n)
    xm_n = torch.empty(cb.cbw_mask_words(desc_n), dtype=torch.int32, device=dev)
    dym_n = torch.empty(cb.cbw_dy_mask_words(desc_n), dtype=torch.int32, device=dev)
    cb.cbw_relu_mask_pack(desc_n, x_n, xm_n)
    cb.cbw_nonzero_mask_pack(desc_n.dtype, dy_n.numel(), dy_n, dym_n)
    ws_mn = cb.workspace(desc_n, cb.CBW_OP_BWD_DATA_MASKED, dev)
    ws_wn = cb.workspace(desc_n, cb.CBW_OP_BWD_WEIGHT, dev)

    def sparse_step_nchw():
        cb.conv_bwd_data_masked(desc_n, dy_n, w, xm_n, dx_n, ws_mn, 0)
        cb.conv_bwd_weight_sparse(desc_n, x_n, dy_n, dym_n, dw, ws_wn, 0)

    for _ in range(20):
        sparse_step_nchw()
    ms_nchw, _ = timed(sparse_step_nchw, args.steps)
    del x_n, dy_n, dx_n, xm_n, dym_n, ws_mn, ws_wn

    # The largest configuration: the whole VGG-16 conv stack (13 layers,
    # N = 32 at 224 x 224), inputs drawn on the device with the same recipe.
    stack = None
    if not args.no_stack:
        log("VGG-16 stack (13 layers), inputs drawn on the device")
        stack = vgg16_stack(cb, torch, max(3, args.steps // 4), args.rounds)

    # Context only: the same dense backward through torch's convolution
    # backward (MIOpen), on the same tensors viewed as channels-last NCHW.
    miopen = gemm_ctx = None
    if not args.no_context:
        log("timing the dense backward through torch (MIOpen), context only")
        try:
            xv, wv, dyv = x.permute(0, 3, 1, 2), w.permute(0, 3, 1, 2), dy.permute(0, 3, 1, 2)

            def miopen_bwd():
                torch.ops.aten.convolution_backward(dyv, xv, wv, None, [spec.stride] * 2, [spec.pad] * 2, [1, 1],
                                                    False, [0, 0], 1, [True, True, False])

            for _ in range(10):
                miopen_bwd()
            ms_mi, _ = timed(miopen_bwd, max(10, args.steps // 2))
            miopen = {"dense_dx_dw_ms": round(ms_mi, 4), "our_dense_step_speedup": round(ms_mi / ms_dense, 3),
                      "layout": "channels-last bf16", "call": "torch.ops.aten.convolution_backward"}
        except Exception as exc:  # context only: a failure there does not void the measurement
            miopen = {"error": str(exc)[:200]}
        # Context only: plain library GEMMs (hipBLASLt through torch.matmul) of
        # the two gradients' GEMM shapes with the same FLOP count (no im2col,
        # no footprint), and a large square one, the practical matrix-core
        # rate of the library on this GPU.
        log("timing plain library GEMMs, context only")
        try:
            gemm_ctx = {}
            npq, crs = spec.N * desc.P * desc.Q, spec.C * spec.R * spec.S
            for name, (m, k, n) in (("dx_shape", (npq, spec.K * spec.R * spec.S, spec.C)),
                                    ("dw_shape", (spec.K, npq, crs)), ("square_8192", (8192, 8192, 8192))):
                a_m = torch.randn(m, k, device=dev).to(torch.bfloat16)
                b_m = torch.randn(k, n, device=dev).to(torch.bfloat16)

                def mm():
                    torch.matmul(a_m, b_m)

                for _ in range(10):
                    mm()
                ms_mm, _ = timed(mm, 20)
                gemm_ctx[name] = {"mnk": [m, n, k], "ms": round(ms_mm, 4),
                                  "tflops": round(2 * m * n * k / (ms_mm * 1e-3) / 1e12, 1)}
                del a_m, b_m
        except Exception as exc:
            gemm_ctx = {"error": str(exc)[:200]}

    if args.copy_calibration:
        a = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    cpu = None
    if not args.no_cpu:
        log("oracle CPU baseline (~%.0f s)" % args.cpu_seconds)
        cpu = cpu_baseline(spec, t_cpu, args.cpu_seconds)

    out = {
        "metric": "useful & dense-equiv TFLOP/s of masked conv bwd (dX+dW); speedup vs dense",
        "value": round(dense_eq, 2),
        "unit": "TFLOP/s (dense-equivalent)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_sparse, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; stands in for the paper's ImageNet training traces)",
        "config": {"workload": "vgg_conv3x3_N32_C256_K256_56x56_s1p1_bf16",
                   "N": spec.N, "C": spec.C, "K": spec.K, "H": spec.H, "W": spec.W, "R": spec.R, "S": spec.S,
                   "x_density": round(nnz_mask / x.numel(), 4), "dy_density": round(nnz_dy / dy.numel(), 4)},
        "useful_tflops": round(useful, 2),
        "speedup_vs_dense": round(ms_dense / ms_sparse, 4),
        "dense_ms_per_step": round(ms_dense, 4),
        "timing": {"rounds": args.rounds, "steps_per_round": args.steps,
                   "sparse_ms_per_round": [round(v, 4) for v in per_round["sparse"]],
                   "dense_ms_per_round": [round(v, 4) for v in per_round["dense"]],
                   "rule": "median over rounds; sparse and dense alternate, the order flipping every round"},
        "dense_equiv_tflops_dense_path": round(2 * f_conv / (ms_dense * 1e-3) / 1e12, 2),
        "executed_fraction": {"dx_rows": round(exec_frac_dx, 6), "dw_blocks": round(exec_frac_dw, 6)},
        "executed_tflops": round(f_exec / (ms_sparse * 1e-3) / 1e12, 2),
        "kernels_ms": {"dx_launch": round(ms_dx_gemm, 4), "dw_gemm": round(ms_dw_gemm, 4),
                       "dx_launch_dense": round(ms_dx_gemm_dense, 4), "dw_gemm_dense": round(ms_dw_gemm_dense, 4),
                       "step_with_events": round(ms_sparse_k, 4),
                       "note": "dx_launch: the data-gradient GEMM and, in its tail workgroups, the weight "
                               "gradient's split-K reduction"},
        "step_distribution": dist,
        "parity": parity,
        "separate_calls": {"sparse_ms": round(ms_sep_sparse, 4), "dense_ms": round(ms_sep_dense, 4),
                           "speedup_vs_dense": round(ms_sep_dense / ms_sep_sparse, 4),
                           "combined_dense_ms_same_rounds": round(ms_dense_here, 4),
                           "note": "the same step through conv_bwd_data_masked + conv_bwd_weight_sparse "
                                   "(dense: conv_bwd_data + conv_bwd_weight_sparse NO_SKIP), 6-7 and 4 launches"},
        "dense_plus_mask_multiply_ms": round(ms_dense_mask, 4),
        "speedup_vs_dense_plus_mask_multiply": round(ms_dense_mask / ms_sparse, 4),
        "nchw_boundary": {"sparse_step_ms": round(ms_nchw, 4), "added_ms": round(ms_nchw - ms_sparse, 4),
                          "note": "NCHW activations through the boundary transposes; NHWC is native"},
        "vgg16_stack": stack,
        "measured_peaks": peaks,
        "miopen_context": miopen,
        "library_gemm_context": gemm_ctx,
        "mask_pack_ms": round(ms_pack, 4),
        "forward_relu_mask": {"ms": round(ms_fwd, 4), "tflops": round(f_conv / (ms_fwd * 1e-3) / 1e12, 2)},
        "flops": {"dx_dense": f_conv, "dw_dense": f_conv, "dx_useful": f_useful_dx, "dw_useful": f_useful_dw},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "paper_context": "paper reports 1.69x-5.43x backward-pass speedup over its own dense mode on a "
                         "simulated 32nm FP16 ASIC (not comparable hardware)",
    }
    print(json.dumps(out), flush=True)
    if not parity["ok"]:
        log("PARITY FAILURE: %s" % parity)
        sys.exit(1)


def alternate(fns, time_fn, rounds):
    """Time each callable of `fns` once per round with time_fn, rotating the
    order every round (round r starts at entry r mod len, so with two
    entries the order flips).  Returns name -> list of per-round results."""
    names = list(fns)
    out = {n: [] for n in names}
    for r in range(rounds):
        k = r % len(names)
        for n in names[k:] + names[:k]:
            out[n].append(time_fn(fns[n]))
    return out


def check_against_oracle(spec, t, dx, dw, x, nsample=400):
    """Sampled parity of the timed step's dX and dW against the oracle (the
    same normwise bound the tests use), plus the exact zero pattern of dX
    over the whole tensor: every output whose footprint bit is clear must be
    the +0.0 pattern."""
    import numpy as np
    import torch
    import oracle
    rng = np.random.default_rng(771)
    st, pd = (spec.stride,) * 2, (spec.pad,) * 2
    tol = 2e-2 if spec.dtype == "bf16" else 1e-5
    killed_nonzero = int(((dx.view(torch.int16) != 0) & ~(x > 0)).sum().item())
    x64 = oracle.nhwc_to_nchw(t["x"].double().numpy())
    dy64 = oracle.nhwc_to_nchw(t["dy"].double().numpy())
    w64 = oracle.krsc_to_kcrs(t["w"].double().numpy())
    cx = np.stack([rng.integers(0, m, nsample) for m in (spec.N, spec.C, spec.H, spec.W)], 1).astype(np.int32)
    o, _, _ = oracle.conv_bwd_data_at(dy64, w64, (spec.H, spec.W), cx, st, pd)
    live = x64[cx[:, 0], cx[:, 1], cx[:, 2], cx[:, 3]] > 0
    o = np.where(live, o, 0.0)
    g = dx.float().cpu().numpy()[cx[:, 0], cx[:, 2], cx[:, 3], cx[:, 1]].astype(np.float64)
    e_dx = float(np.max(np.abs(g - o)) / max(np.max(np.abs(o)), 1e-300))
    cw = np.stack([rng.integers(0, m, nsample) for m in (spec.K, spec.C, spec.R, spec.S)], 1).astype(np.int32)
    o, _, _ = oracle.conv_bwd_weight_at(x64, dy64, (spec.R, spec.S), cw, st, pd)
    g = dw.cpu().numpy()[cw[:, 0], cw[:, 2], cw[:, 3], cw[:, 1]].astype(np.float64)
    e_dw = float(np.max(np.abs(g - o)) / max(np.max(np.abs(o)), 1e-300))
    ok = killed_nonzero == 0 and e_dx <= tol and e_dw <= tol
    return {"ok": bool(ok), "dx_normwise_err": e_dx, "dw_normwise_err": e_dw, "tol": tol,
            "killed_outputs_not_plus_zero": killed_nonzero, "samples": nsample}


def measure_peaks(torch, stream):
    """Measured ceilings on this GPU: a bf16 matrix-core loop (16x16x32 and
    32x32x16 instructions, four waves per SIMD, no memory traffic) and two
    HBM streams over 1 GiB buffers (4x the last-level cache): read only, and
    copy (bytes read + written).  Best of five launches each."""
    import paper_2109_07710_amd.peaks as pk
    dev = torch.device("cuda:0")
    seed = torch.randn(pk.seed_bytes() // 2, device=dev).to(torch.bfloat16)
    blocks = 256 * 4
    sink = torch.zeros(pk.sink_words(blocks), dtype=torch.int32, device=dev)
    res = {}

    def best(launch, n=5):
        for _ in range(2):
            launch()
        torch.cuda.synchronize()
        ms = []
        for _ in range(n):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            launch()
            b.record(stream)
            torch.cuda.synchronize()
            ms.append(a.elapsed_time(b))
        return min(ms)

    try:
        iters = 8192
        for shape, name in ((pk.MFMA_16X16X32, "16x16x32"), (pk.MFMA_32X32X16, "32x32x16")):
            ms = best(lambda: pk.mfma(shape, blocks, iters, seed, sink, stream))
            res["mfma_bf16_%s_tflops" % name] = round(pk.mfma_flops(shape, blocks, iters) / (ms * 1e-3) / 1e12, 1)
        res["mfma_bf16_tflops"] = max(res["mfma_bf16_16x16x32_tflops"], res["mfma_bf16_32x32x16_tflops"])
        nbytes = 1 << 30
        src = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        ms = best(lambda: pk.hbm_read(src, sink, stream))
        res["hbm_read_gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
        ms = best(lambda: pk.hbm_copy(src, dst, stream))
        res["hbm_copy_gbs"] = round(2 * nbytes / (ms * 1e-3) / 1e9, 1)
        del src, dst
        res["spec"] = {"mfma_bf16_tflops": PEAK_BF16_TFLOPS, "hbm_gbs": PEAK_HBM_GBS}
        res["method"] = ("bf16 matrix loop: %d workgroups of 4 waves, %d rounds of 8 (16x16x32) or 4 (32x32x16) "
                         "independent instructions per wave; HBM: 1 GiB streams; best of 5" % (blocks, iters))
    except Exception as exc:  # the measurement is context: a failure leaves the spec peaks
        res["error"] = str(exc)[:200]
    return res


def vgg16_stack(cb, torch, steps, rounds):
    """The VGG-16 conv stack (13 layers, N = 32, 224 x 224 input) as one
    step: every layer's sparse backward through conv_bwd_sparse (masked dX
    where the footprint applies, dense dX after a pool, no dX for conv1_1;
    skipping dW), against the same layers' dense step (the same call with no
    footprint and CBW_FLAG_NO_SKIP) and the sparse step through the separate
    calls.  Inputs drawn on the device (workloads.draw_on_device, same recipe
    as the tests)."""
    import numpy as np
    import workloads as wl
    dev = torch.device("cuda:0")
    layers = []
    for spec in wl.config5():
        t = wl.draw_on_device(spec, dev)
        x, w, dy = t["x"], t["w"], t["dy"]
        desc = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad)
        L = {"spec": spec, "desc": desc, "x": x, "w": w, "dy": dy,
             "xm": torch.empty(cb.cbw_mask_words(desc), dtype=torch.int32, device=dev),
             "dym": torch.empty(cb.cbw_dy_mask_words(desc), dtype=torch.int32, device=dev),
             "dx": torch.empty_like(x) if spec.need_dx else None,
             "dw": torch.empty((spec.K, spec.R, spec.S, spec.C), dtype=torch.float32, device=dev),
             "ws_m": cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED, dev) if spec.need_dx and spec.masked else None,
             "ws_d": cb.workspace(desc, cb.CBW_OP_BWD_DATA, dev) if spec.need_dx else None,
             "ws_w": cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT, dev),
             "ws_b": cb.workspace(desc, cb.CBW_OP_BWD_BOTH, dev)}
        cb.cbw_relu_mask_pack(desc, x, L["xm"])
        cb.cbw_nonzero_mask_pack(desc.dtype, dy.numel(), dy, L["dym"])
        true_c = spec.extra.get("true_c", spec.C)
        L["useful"] = 2 * int(torch.count_nonzero(dy).item()) * true_c * spec.R * spec.S
        L["dense_flops"] = spec.dense_flops() * (2 if spec.need_dx else 1)
        if spec.need_dx:
            L["useful"] += (2 * int(torch.count_nonzero(x > 0).item()) * spec.K * spec.R * spec.S
                            if spec.masked else spec.dense_flops())
        layers.append(L)

    def sparse(L):
        s = L["spec"]
        cb.conv_bwd_sparse(L["desc"], L["x"], L["dy"], L["w"], L["xm"] if s.need_dx and s.masked else None,
                           L["dym"], L["dx"], L["dw"], L["ws_b"], 0)

    def dense(L):
        cb.conv_bwd_sparse(L["desc"], L["x"], L["dy"], L["w"], None, None, L["dx"], L["dw"], L["ws_b"],
                           cb.CBW_FLAG_NO_SKIP)

    def separate(L):
        d, s = L["desc"], L["spec"]
        if s.need_dx:
            if s.masked:
                cb.conv_bwd_data_masked(d, L["dy"], L["w"], L["xm"], L["dx"], L["ws_m"], 0)
            else:
                cb.conv_bwd_data(d, L["dy"], L["w"], L["dx"], L["ws_d"])
        cb.conv_bwd_weight_sparse(d, L["x"], L["dy"], L["dym"], L["dw"], L["ws_w"], 0)

    def tm(fn):
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    kinds = {"sparse": sparse, "dense": dense, "separate": separate}
    for _ in range(3):
        for fn in kinds.values():
            for L in layers:
                fn(L)
    whole = alternate({k: (lambda f=f: [f(L) for L in layers]) for k, f in kinds.items()}, tm, rounds)
    res = {k: float(np.median(v)) for k, v in whole.items()}
    per_layer = []
    for L in layers:
        r = alternate({k: (lambda f=f, L=L: f(L)) for k, f in kinds.items()}, tm, 3)
        s = L["spec"]
        per_layer.append({"layer": s.name, "C": s.extra.get("true_c", s.C), "K": s.K, "HW": s.H,
                          "dx": "masked" if s.need_dx and s.masked else ("dense" if s.need_dx else "none"),
                          **{k + "_ms": round(float(np.median(v)), 4) for k, v in r.items()}})
    useful = sum(L["useful"] for L in layers)
    dense_flops = sum(L["dense_flops"] for L in layers)
    out = {"sparse_ms": round(res["sparse"], 4), "dense_ms": round(res["dense"], 4),
           "separate_calls_ms": round(res["separate"], 4),
           "speedup_vs_dense": round(res["dense"] / res["sparse"], 4),
           "separate_calls_speedup_vs_dense": round(res["dense"] / res["separate"], 4),
           "dense_equiv_tflops": round(dense_flops / (res["sparse"] * 1e-3) / 1e12, 2),
           "useful_tflops": round(useful / (res["sparse"] * 1e-3) / 1e12, 2),
           "dense_gflop": round(dense_flops / 1e9, 1), "useful_gflop": round(useful / 1e9, 1),
           "steps_per_round": steps, "rounds": rounds, "layers": per_layer,
           "inputs": "drawn on the device (workloads.draw_on_device), N=32, 224x224"}
    del layers
    torch.cuda.empty_cache()
    return out


def layer_timing(cb, torch, spec, steps, warmup):
    """Sparse and dense step times of one layer (same schedule as the main
    line) plus the kernels' executed fractions."""
    import workloads as wl
    dev = torch.device("cuda:0")
    t = wl.draw(spec)
    x, w, dy = (t[k].to(dev) for k in ("x", "w", "dy"))
    del t
    desc = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad)
    xm = torch.empty(cb.cbw_mask_words(desc), dtype=torch.int32, device=dev)
    dym = torch.empty(cb.cbw_dy_mask_words(desc), dtype=torch.int32, device=dev)
    cb.cbw_relu_mask_pack(desc, x, xm)
    cb.cbw_nonzero_mask_pack(desc.dtype, dy.numel(), dy, dym)
    dx = torch.empty_like(x)
    dw = torch.empty((spec.K, spec.R, spec.S, spec.C), dtype=torch.float32, device=dev)
    ws_m = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED, dev)
    ws_d = cb.workspace(desc, cb.CBW_OP_BWD_DATA, dev)
    ws_w = cb.workspace(desc, cb.CBW_OP_BWD_WEIGHT, dev)
    ws_b = cb.workspace(desc, cb.CBW_OP_BWD_BOTH, dev)
    b_off = cb.both_weight_offset(desc)
    masked_dx = spec.need_dx and spec.masked

    # The step of the main line: one conv_bwd_sparse call (dX masked where
    # the layer's data gradient is, dense where it is not, none for a first
    # layer); the dense step is the same call without footprints and NO_SKIP.
    def sparse():
        cb.conv_bwd_sparse(desc, x, dy, w, xm if masked_dx else None, dym, dx if spec.need_dx else None, dw,
                           ws_b, 0)

    def dense():
        cb.conv_bwd_sparse(desc, x, dy, w, None, None, dx if spec.need_dx else None, dw, ws_b,
                           cb.CBW_FLAG_NO_SKIP)

    # the same step through the separate entry points
    def separate():
        if spec.need_dx:
            if spec.masked:
                cb.conv_bwd_data_masked(desc, dy, w, xm, dx, ws_m, 0)
            else:
                cb.conv_bwd_data(desc, dy, w, dx, ws_d)
        cb.conv_bwd_weight_sparse(desc, x, dy, dym, dw, ws_w, 0)

    def sparse_x():
        # as sparse(), with the weight gradient also skipping all-zero X blocks
        if spec.need_dx:
            if spec.masked:
                cb.conv_bwd_data_masked(desc, dy, w, xm, dx, ws_m, 0)
            else:
                cb.conv_bwd_data(desc, dy, w, dx, ws_d)
        cb.conv_bwd_weight_sparse_x(desc, x, dy, xm, dym, dw, ws_w, 0)

    def tm(fn):
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps

    # The steps are warmed up together (the clocks ramp up after the host-side
    # input generation), then timed in alternating rounds; medians count.
    for _ in range(warmup):
        sparse()
        sparse_x()
        dense()
        separate()
    import numpy as np
    rr = alternate({"s": sparse, "x": sparse_x, "d": dense, "p": separate}, tm, 3)
    ms_s, ms_x, ms_d, ms_p = (float(np.median(rr[k])) for k in ("s", "x", "d", "p"))
    sparse_x()
    st_x = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws_w)
    work_x = cb.cbw_read_weight_work(desc, ws_w)
    separate()
    sparse()
    torch.cuda.synchronize()
    work = cb.cbw_read_weight_work(desc, ws_b[b_off:])
    rec = {"layer": spec.name, "N": spec.N, "C": spec.C, "K": spec.K, "H": spec.H, "W": spec.W, "R": spec.R,
           "masked_dx": bool(spec.need_dx and spec.masked), "need_dx": bool(spec.need_dx),
           "x_density": round(float((x > 0).float().mean().item()), 4),
           "dy_density": round(float((dy != 0).float().mean().item()), 4),
           "sparse_ms": round(ms_s, 4), "dense_ms": round(ms_d, 4), "speedup_vs_dense": round(ms_d / ms_s, 4),
           "separate_calls_ms": round(ms_p, 4)}
    f = spec.dense_flops()
    nflops = f * (2 if spec.need_dx else 1)
    rec["dense_equiv_tflops"] = round(nflops / (ms_s * 1e-3) / 1e12, 2)
    # HBM roofline: the algorithmic bytes of the step against 8 TB/s (the
    # bound for the 1x1 layers, whose arithmetic intensity is far below the
    # ridge) next to the matrix-core floor of its dense-equivalent FLOPs
    nbytes = step_bytes(spec)
    rec["algorithmic_mb"] = round(nbytes / 1e6, 2)
    rec["hbm_floor_ms"] = round(nbytes / (PEAK_HBM_GBS * 1e9) * 1e3, 4)
    rec["mfma_floor_ms"] = round(nflops / (PEAK_BF16_TFLOPS * 1e12) * 1e3, 4)
    rec["bound"] = "hbm" if rec["hbm_floor_ms"] > rec["mfma_floor_ms"] else "mfma"
    rec["hbm_frac"] = round(rec["hbm_floor_ms"] / ms_s, 4)
    rec["mfma_frac_dense_equiv"] = round(rec["mfma_floor_ms"] / ms_s, 4)
    useful = 2 * int(torch.count_nonzero(dy).item()) * spec.extra.get("true_c", spec.C) * spec.R * spec.S
    if spec.need_dx:
        useful += (2 * int(torch.count_nonzero(x > 0).item()) * spec.K * spec.R * spec.S if spec.masked else f)
    rec["useful_tflops"] = round(useful / (ms_s * 1e-3) / 1e12, 2)
    if spec.need_dx and spec.masked:
        st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_DATA_MASKED, ws_b)
        rec["dx_rows_executed"] = round(st.rows_live / st.rows_total, 4)
    st = cb.cbw_read_stats(desc, cb.CBW_OP_BWD_WEIGHT, ws_b[b_off:])
    rec["dw_blocks_executed"] = round(1.0 - st.blocks_skipped / max(st.blocks_total, 1), 4)
    rec["dw_split_balance"] = split_balance(work)
    # the variant whose weight gradient also skips all-zero X blocks
    rec["sparse_x_ms"] = round(ms_x, 4)
    rec["speedup_x_vs_dense"] = round(ms_d / ms_x, 4)
    rec["dw_blocks_executed_x"] = round(1.0 - st_x.blocks_skipped / max(st_x.blocks_total, 1), 4)
    rec["dw_split_balance_x"] = split_balance(work_x)
    # the per-layer dispatch of the main line, decided from the stats above
    st_dx = (cb.cbw_read_stats(desc, cb.CBW_OP_BWD_DATA_MASKED, ws_m)
             if spec.need_dx and spec.masked else None)
    dx_skip, dw_skip = adaptive_choice(st_dx, st)

    def adaptive():
        if spec.need_dx:
            if spec.masked:
                cb.conv_bwd_data_masked(desc, dy, w, xm, dx, ws_m, 0 if dx_skip else cb.CBW_FLAG_NO_SKIP)
            else:
                cb.conv_bwd_data(desc, dy, w, dx, ws_d)
        if dw_skip:
            cb.conv_bwd_weight_sparse(desc, x, dy, dym, dw, ws_w, 0)
        else:
            cb.conv_bwd_weight_sparse(desc, x, dy, None, dw, ws_w, cb.CBW_FLAG_NO_SKIP)

    for _ in range(max(warmup // 4, 2)):
        adaptive()
    ra = alternate({"a": adaptive, "d": dense}, tm, 3)
    ms_a = float(np.median(ra["a"]))
    rec["adaptive_ms"] = round(ms_a, 4)
    rec["speedup_adaptive_vs_dense"] = round(ms_d / ms_a, 4)
    rec["adaptive_calls"] = "dX %s, dW %s" % ("compacting" if dx_skip else "non-skipping",
                                              "skipping" if dw_skip else "non-skipping")
    return rec


def step_bytes(spec):
    """Algorithmic HBM bytes of one backward step of a layer: every operand
    read once and every result written once (dX: dY, W, the footprint bits
    when masked, dX; dW: X, dY, dW in fp32)."""
    e = 2 if spec.dtype == "bf16" else 4
    npix, npq = spec.N * spec.H * spec.W, spec.N * spec.P * spec.Q
    b = npix * spec.C * e + npq * spec.K * e + spec.K * spec.R * spec.S * spec.C * 4
    if spec.need_dx:
        b += npq * spec.K * e + spec.K * spec.R * spec.S * spec.C * e + npix * spec.C * e
        if spec.masked:
            b += (npix * spec.C + 7) // 8
    return b


def adaptive_choice(st_dx, st_dw):
    """Per-layer dispatch from an earlier call's statistics (None: no data
    gradient): compact the data gradient when at most 90% of its pixel rows
    were live, skip weight-gradient blocks when at least 5% were skippable."""
    dx_skip = st_dx is not None and st_dx.rows_live <= 0.9 * st_dx.rows_total
    dw_skip = st_dw.blocks_skipped >= 0.05 * max(st_dw.blocks_total, 1)
    return dx_skip, dw_skip


def split_balance(work):
    """Executed weight-gradient blocks over what the busiest split of each
    tile bounds (nsplit x its maximum), summed over the tiles: 1.0 when every
    split of a tile executes the same number of blocks."""
    cap = int(work.max(axis=0).sum()) * work.shape[0]
    return round(int(work.sum()) / cap, 4) if cap else 1.0


def elementwise_sweep(args):
    """Break-even of the per-element data gradient (vector ALUs, every zero dY
    entry and every dead pixel skipped) against the matrix-core masked path,
    data gradient only, on i.i.d. footprints with mask density = dY density
    = d (configuration 4's layer and configuration 2's layer)."""
    import torch
    import paper_2109_07710_amd as cb
    import workloads as wl
    dev = torch.device("cuda:0")
    for make, tag in ((lambda d: wl.config4(d, "bernoulli")[0], "conv3x3_c512_14x14_N128"),
                      (lambda d: wl.LayerSpec("vgg_conv3x3_c256_56x56", 2, 0, N=32, C=256, H=56, W=56, K=256, R=3, S=3,
                                              x_kind="shifted_gauss", x_param=wl.threshold_for_density(d),
                                              dy_kind="bernoulli", dy_param=d), "conv3x3_c256_56x56_N32")):
        for d in (0.01, 0.02, 0.03, 0.05, 0.1, 0.2, 0.4):
            spec = make(d)
            log("elementwise sweep %s d=%.2f" % (tag, d))
            t = wl.draw(spec)
            x, w, dy = (t[k].to(dev) for k in ("x", "w", "dy"))
            del t
            desc = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad)
            xm = torch.zeros(cb.cbw_mask_words(desc), dtype=torch.int32, device=dev)
            cb.cbw_relu_mask_pack(desc, x, xm)
            dx = torch.empty_like(x)
            ws_m = cb.workspace(desc, cb.CBW_OP_BWD_DATA_MASKED, dev)
            ws_e = cb.workspace(desc, cb.CBW_OP_BWD_DATA_ELEMENTWISE, dev)

            def mfma():
                cb.conv_bwd_data_masked(desc, dy, w, xm, dx, ws_m, 0)

            def valu():
                cb.conv_bwd_data_elementwise(desc, dy, w, xm, dx, ws_e)

            def tm(fn, n):
                torch.cuda.synchronize()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for _ in range(n):
                    fn()
                b.record()
                torch.cuda.synchronize()
                return a.elapsed_time(b) / n

            for _ in range(10):
                mfma()
                valu()
            ms_m, ms_v = float("inf"), float("inf")
            for _ in range(2):
                ms_m = min(ms_m, tm(mfma, 10))
                ms_v = min(ms_v, tm(valu, 10))
            _, products = cb.cbw_read_pixel_counts(desc, ws_e)
            f_useful = 2 * int(useful_products(x, dy, spec))
            print(json.dumps({"sweep": "elementwise", "layer": tag, "density": d,
                              "mfma_masked_dx_ms": round(ms_m, 4), "valu_elementwise_dx_ms": round(ms_v, 4),
                              "valu_over_mfma": round(ms_v / ms_m, 3),
                              "valu_products_executed": products,
                              "valu_executed_gflop": round(2 * products * spec.C / 1e9, 3),
                              "useful_gflop": round(f_useful / 1e9, 3),
                              "dense_gflop": round(spec.dense_flops() / 1e9, 3)}), flush=True)
            del x, w, dy, xm, dx, ws_m, ws_e


def useful_products(x, dy, spec):
    """Multiply-adds of the data gradient that have a live output and a
    non-zero dY operand (IN+OUT useful work), counted on the device from the
    tensors: for each output pixel, live channels x non-zero dY entries over
    its in-range taps (stride 1)."""
    import torch
    live_c = (x > 0).sum(dim=3).double()                      # [N,H,W] live channels per pixel
    nz = (dy != 0).sum(dim=3).double()                        # [N,P,Q] non-zeros per source pixel
    pad = torch.nn.functional.pad(nz, (spec.pad, spec.pad, spec.pad, spec.pad))
    tot = torch.zeros_like(live_c)
    for r in range(spec.R):
        for s in range(spec.S):
            # output (h, w) reads source (h + pad - r, w + pad - s)
            tot += pad[:, 2 * spec.pad - r:2 * spec.pad - r + spec.H, 2 * spec.pad - s:2 * spec.pad - s + spec.W]
    return (tot * live_c).sum().item()


def trace_layer(args):
    """One layer's combined sparse step (footprints as the workload defines
    them) and dense step, in alternating rounds: round r runs `--steps`
    calls of one step after a one-element fill kernel (the marker a trace
    parser splits phases at).  Layers: the configuration-2 layer, the three
    bottleneck layers, the 13 VGG-16 layers."""
    import numpy as np
    import torch
    import paper_2109_07710_amd as cb
    import workloads as wl
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    specs = {s.name: s for s in wl.config2() + wl.config3() + wl.config5()}
    if args.trace_layer not in specs:
        print("unknown layer %r; one of: %s" % (args.trace_layer, ", ".join(sorted(specs))), file=sys.stderr)
        sys.exit(2)
    spec = specs[args.trace_layer]
    t = wl.draw_on_device(spec, dev) if spec.config_id == 5 else {k: v.to(dev) for k, v in wl.draw(spec).items()}
    x, w, dy = t["x"], t["w"], t["dy"]
    desc = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad)
    xm = torch.empty(max(cb.cbw_mask_words(desc), 1), dtype=torch.int32, device=dev)
    dym = torch.empty(max(cb.cbw_dy_mask_words(desc), 1), dtype=torch.int32, device=dev)
    cb.cbw_relu_mask_pack(desc, x, xm)
    cb.cbw_nonzero_mask_pack(desc.dtype, dy.numel(), dy, dym)
    dx = torch.empty_like(x) if spec.need_dx else None
    dw = torch.empty((spec.K, spec.R, spec.S, spec.C), dtype=torch.float32, device=dev)
    ws = cb.workspace(desc, cb.CBW_OP_BWD_BOTH, dev)
    masked_dx = spec.need_dx and spec.masked
    steps = {"sparse": lambda: cb.conv_bwd_sparse(desc, x, dy, w, xm if masked_dx else None, dym, dx, dw, ws, 0),
             "dense": lambda: cb.conv_bwd_sparse(desc, x, dy, w, None, None, dx, dw, ws, cb.CBW_FLAG_NO_SKIP)}
    marker = torch.empty(1, device=dev)
    for _ in range(args.warmup):
        steps["sparse"]()
        steps["dense"]()
    torch.cuda.synchronize()
    order, times = [], {k: [] for k in steps}
    for r in range(args.rounds):
        for name in (("sparse", "dense") if r % 2 == 0 else ("dense", "sparse")):
            marker.fill_(float(len(order)))
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(args.steps):
                steps[name]()
            b.record()
            torch.cuda.synchronize()
            order.append(name)
            times[name].append(a.elapsed_time(b) / args.steps)
    if args.copy_calibration:
        # the byte counters' reference: a plain copy of 256 MiB, three times
        src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
    print(json.dumps({"trace_layer": spec.name, "steps_per_round": args.steps, "order": order,
                      "ms_per_step_median": {k: round(float(np.median(v)), 4) for k, v in times.items()}}),
          flush=True)


def run_sweep(args):
    import torch
    if args.sweep == "elementwise":
        return elementwise_sweep(args)

    import paper_2109_07710_amd as cb
    import workloads as wl
    torch.cuda.set_device(0)
    if args.sweep == "config4":
        specs = [(kind, wl.config4(d, kind)[0]) for kind in ("bernoulli", "clustered", "channel_shared")
                 for d in wl.SWEEP_DENSITIES]
    elif args.sweep == "config3":
        specs = [("bottleneck", s) for s in wl.config3()]
    elif args.sweep == "config5":
        specs = [("vgg16", s) for s in wl.config5()]
    else:
        # the four post-pool layers with their data gradient masked by pooled > 0
        specs = [("vgg16_pooled_mask", s) for s in wl.config5(pooled_mask=True) if s.layer_id in (3, 5, 8, 11)]
    for tag, spec in specs:
        d = cb.ConvDesc.make(spec.N, spec.C, spec.H, spec.W, spec.K, spec.R, spec.S, spec.stride, spec.pad)
        if cb.cbw_validate_desc(d) != cb.CBW_OK:
            print(json.dumps({"sweep": args.sweep, "kind": tag, "layer": spec.name,
                              "skipped": "unsupported by the library (channel count)"}), flush=True)
            continue
        log("sweep point %s %s" % (tag, spec.name))
        rec = layer_timing(cb, torch, spec, max(5, args.steps // 2), 25)
        rec = {"sweep": args.sweep, "kind": tag, **rec}
        if "density" in spec.extra:
            rec["density"] = spec.extra["density"]
        print(json.dumps(rec), flush=True)


def traffic_for(kernel):
    """HBM bytes per launch measured by rocprofv3 FETCH_SIZE/WRITE_SIZE
    counters (profiles/hbm_traffic_config2.json), or None when absent or taken
    from a different kernel source than the one built now."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "hbm_traffic_config2.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    entry = rec.get(kernel)
    if not entry or not entry.get("sources"):
        return None
    h = hashlib.sha256()
    for src in entry["sources"]:
        h.update(open(os.path.join(ROOT, src), "rb").read())
    if entry.get("sources_sha256") != h.hexdigest():
        return None
    return entry.get("hbm_bytes_per_launch")


def cpu_baseline(spec, t, budget_s):
    """The oracle (fp64 direct loops, OpenMP) on whole images of the same
    layer until the time budget is spent; throughput in the same
    dense-equivalent TFLOP/s."""
    import oracle
    w64 = oracle.krsc_to_kcrs(t["w"].double().numpy())
    st, pd = (spec.stride,) * 2, (spec.pad,) * 2
    done, el = 0, 0.0
    while done < spec.N and el < budget_s:
        x64 = oracle.nhwc_to_nchw(t["x"][done:done + 1].double().numpy())
        dy64 = oracle.nhwc_to_nchw(t["dy"][done:done + 1].double().numpy())
        mask = oracle.relu_mask(x64)
        t0 = time.perf_counter()
        oracle.conv_bwd_data(dy64, w64, (spec.H, spec.W), st, pd, mask=mask)
        oracle.conv_bwd_weight(x64, dy64, (spec.R, spec.S), st, pd)
        el += time.perf_counter() - t0
        done += 1
    flops = 2 * spec.dense_flops() * done / spec.N
    return {"value": round(flops / el / 1e12, 6), "unit": "TFLOP/s (dense-equivalent)",
            "cores": oracle.num_threads(), "kind": "oracle", "cpu": cpu_model(),
            "gmac_per_s": round(flops / 2 / el / 1e9, 3),
            "sample": "%d of %d images of the same layer (masked dX + dW, fp64), %.1f s" % (done, spec.N, el)}


def cpu_model():
    """The host CPU's model name (Linux), or the platform's processor string."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


if __name__ == "__main__":
    main()
