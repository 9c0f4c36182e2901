#!/usr/bin/env python3
"""Benchmark of the CCI-sparse forward path on one MI355X.

One step = the whole hot path over one batch of synthetic input: cci_pack
(per-group top-K of the dense fp32 master weights -> packed bf16 values +
uint8 indices) followed by the CCI-sparse product (fp32 accumulation, bf16
out).

Default workload: the sparsity-sweep FC layer, X bf16 [4096, 4096] ~ N(0,1),
W [4096, 4096] ~ N(0, 1/4096), G = 16.  `value` is the step at K = 4 (75%
sparse; --k picks another); the same line carries every K of the sweep
{1, 2, 4, 8, 16} (K = 16 is the dense control) under `sweep_k`: product time,
effective TFLOP/s, roofline fraction, hipBLASLt bf16 GEMM time on the same
rotated X and the speedup.

Metric: effective TFLOP/s = 2 * N * nnz / step time (N rows, nnz kept
weights).  Inputs are resident in HBM before timing starts; X and Y rotate
over enough copies (> 2x the 256 MB last-level cache) that no step reads its
activations from cache.

Roofline of the product kernel: the method's own work -- algorithmic bytes
(X once, packed weights once, Y once) against 8 TB/s and 2 * N * nnz flop
against the 2516.6 TFLOP/s bf16 matrix-core peak, whichever takes longer.
The matrix cores actually execute the product of the expanded dense tile
(2 * N * C * O flop); that utilisation is reported separately as
`mfma_expanded_util`.

`--workload NAME` runs the same contract on another configuration (conv3x3,
conv1x1_k4, ...); `--sweep` prints one line per configuration.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

# HBM and dense bf16 matrix-core peaks as published; the vector peak is the
# fp32 FMA rate without packed math (256 CUs x 4 SIMDs x 16 lanes x 2 flop x
# 2.4 GHz): the kernels are built with packed-fp32 instruction selection off.
PEAK = {"hbm_GBps": 8000.0, "mfma_bf16_TFLOPs": 2516.6, "valu_fp32_TFLOPs": 78.6}


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="fc4096",
                   help="fc4096 (the K sweep; default) or one named workload (conv3x3, conv1x1_k4, fc4096_k1, ...)")
    p.add_argument("--k", type=int, default=4, help="fc4096: the K whose step gives `value`")
    p.add_argument("--algo", default="auto", choices=["auto", "sparse_mac", "dense_tile_mfma", "wide_tile_mfma", "narrow_mfma",
                                                     "resident_mfma", "few_rows_mfma", "tap_tile_mfma",
                                                     "stream_tile_mfma", "split_k_mfma"])
    p.add_argument("--rotate-mb", type=float, default=600.0,
                   help="total size of rotated X/Y copies (0: no rotation)")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="target wall time of the CPU oracle sample")
    p.add_argument("--no-cpu-configs", action="store_true",
                   help="skip the per-configuration oracle timings (1 core and all cores) of the smaller configs")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-dense", action="store_true")
    p.add_argument("--no-bbs", action="store_true", help="fc4096: skip the balanced-sparsity (2:4) comparison")
    p.add_argument("--no-td", action="store_true", help="fc4096: skip the targeted-dropout training-step kernels")
    p.add_argument("--no-smalln", action="store_true", help="fc4096: skip the few-row (log2 G-bit index) products")
    p.add_argument("--graph", action="store_true",
                   help="replay the timed steps from HIP graphs of 8 steps instead of launching every kernel "
                        "from Python")
    p.add_argument("--sweep", action="store_true",
                   help="instead of the headline line: one JSON line per configuration (FC, 1x1, 3x3, "
                        "FC K-sweep, ResNet-50 forward) with CCI and dense bf16 times")
    p.add_argument("--sweep-only", default="",
                   help="comma-separated subset of the sweep: config names, 'resnet50', 'mobilenetv2'")
    p.add_argument("--mbv2-k", default="1,2,3,4", help="kept weights per group of the MobileNetV2 sweep lines")
    p.add_argument("--calibrate-copy-mb", type=float, default=0.0,
                   help="only run a plain device copy of this many MB (x5) and exit: the reference "
                        "kernel for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes")
    return p.parse_args()


KERNEL_SOURCES = {"cci_dense_tile": "cci_dense_tile.hip", "cci_wide_tile": "cci_wide_tile.hip",
                  "cci_sparse_mac": "cci_sparse_mac.hip", "cci_narrow": "cci_narrow.hip",
                  "cci_resident": "cci_resident.hip", "cci_bits": "cci_bits.hip",
                  "cci_tap_tile": "cci_tap_tile.hip", "cci_stream_tile": "cci_stream_tile.hip",
                  "cci_split_k": "cci_split_k.hip"}


def kernel_source_hash(kernel: str = "cci_dense_tile") -> str:
    """Hash of one kernel's source file with comments and blank space
    removed, so that counter files stay matched to the code they measured
    across edits of comments or of other kernels."""
    h = hashlib.sha256()
    f = KERNEL_SOURCES[kernel]
    with open(os.path.join(HERE, "paper_1910_11971_amd", "csrc", f)) as fh:
        text = re.sub(r"//[^\n]*", "", fh.read())
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    h.update(f.encode() + " ".join(text.split()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload: str, kernel: str, src_hash: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources."""
    path = os.path.join(HERE, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_hash") != src_hash:
        return None
    return d.get("hbm_bytes_per_launch")


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the CCI product shards by rows or by output groups with no "
              "exchange, and only the one-GPU kernel is implemented. Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1910_11971_amd import cci, workloads

    if args.calibrate_copy_mb > 0:
        n = int(args.calibrate_copy_mb * 1e6) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes_each_way": n * 4, "launches": 5}), flush=True)
        return

    if args.sweep:
        return sweep(args)
    if args.workload == "fc4096":
        return main_fc_sweep(args)

    wl = workloads.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    X_cpu, W_np = workloads.draw(wl)
    xdt = torch.bfloat16 if wl.x_dtype == "bf16" else torch.float32
    ydt = torch.bfloat16 if wl.y_dtype == "bf16" else torch.float32
    vdt = xdt
    stride, pad = (wl.stride, wl.stride), (wl.pad, wl.pad)

    # ---- resident inputs, rotated copies --------------------------------------
    x_bytes = X_cpu.numel() * X_cpu.element_size()
    y_bytes = wl.N * wl.O * (2 if ydt == torch.bfloat16 else 4)
    ncopy = 1 if args.rotate_mb <= 0 else max(1, int(np.ceil(args.rotate_mb * 1e6 / (x_bytes + y_bytes))))
    X0 = X_cpu.to(dev)
    Xs = [X0] + [X0.clone() for _ in range(ncopy - 1)]
    yshape = (wl.B, wl.Ho, wl.Wo, wl.O) if wl.conv else (wl.N, wl.O)
    Ys = [torch.empty(yshape, dtype=ydt, device=dev) for _ in range(ncopy)]
    W = torch.from_numpy(W_np).to(dev)
    vals = torch.empty((wl.O // wl.G, wl.K, wl.C), dtype=vdt, device=dev)
    idx = torch.empty((wl.O // wl.G, wl.K, wl.C), dtype=torch.uint8, device=dev)

    stream = torch.cuda.Stream(device=dev)  # default priority
    algo = args.algo if args.algo != "auto" else cci.auto_algo(xdt, vdt, wl.N, wl.C, wl.Cin, wl.O, wl.G, wl.K)

    def conv_only(i):  # the product (a convolution, or an FC layer via cci_spmm)
        if wl.conv:
            cci.conv_im2col(Xs[i % ncopy], vals, idx, wl.G, wl.KH, wl.KW, stride, pad, out_dtype=ydt, algo=algo,
                            out=Ys[i % ncopy])
        else:
            cci.spmm(Xs[i % ncopy], vals, idx, wl.G, out_dtype=ydt, algo=algo, out=Ys[i % ncopy])

    def step(i):
        cci.pack(W, wl.G, wl.K, vdt, out=(vals, idx))
        conv_only(i)

    def pack_only(i):
        cci.pack(W, wl.G, wl.K, vdt, out=(vals, idx))

    # Steps are launched from Python; with --graph they are replayed from HIP
    # graphs of 8 consecutive steps (the rotation has a multiple of 8 copies).
    chunk = 8
    ncopy_g = ncopy
    graphs = {}

    def run_steps(i0, n):
        i = i0
        while i < i0 + n:
            if args.graph and (i % ncopy_g) % chunk == 0 and i + chunk <= i0 + n and ncopy_g % chunk == 0:
                graphs[(i % ncopy_g) // chunk].replay()
                i += chunk
            else:
                step(i)
                i += 1

    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            step(i)
        pack_only(0)
        torch.cuda.synchronize()
    if args.graph and ncopy_g % chunk == 0:
        for gi in range(ncopy_g // chunk):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                for i in range(gi * chunk, (gi + 1) * chunk):
                    step(i)
            graphs[gi] = g
        torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        run_steps(0, ncopy_g)  # replay every graph once before timing
        torch.cuda.synchronize()
        # timed region: K whole steps (pack + conv), nothing else on the stream
        t0 = time.perf_counter()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        run_steps(0, args.steps)
        b.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms_step = a.elapsed_time(b) / args.steps
    # each kernel alone, the same number of launches back to back (graph replays)
    conv_avg = _graph_time(conv_only, ncopy_g, max(1, args.steps // ncopy_g), stream)
    pack_avg = _graph_time(pack_only, 16, max(1, args.steps // 16), stream)

    flop = 2.0 * wl.N * wl.nnz
    value = flop / (ms_step * 1e-3) / 1e12

    # ---- roofline of the dominant kernel (the product) -------------------------
    val_b = 2 if vdt == torch.bfloat16 else 4
    alg_bytes = x_bytes + wl.nnz * (val_b + 1) + y_bytes
    dense_flop = 2.0 * wl.N * wl.C * wl.O
    kname = kernel_name(algo)
    src_hash = kernel_source_hash(kname)
    roof = roof_for(kname, flop, dense_flop, alg_bytes, conv_avg)
    roof["traffic"] = load_traffic(args.workload, kname, src_hash)
    roof["kernel"] = kname
    roof["kernel_avg_us"] = round(conv_avg * 1e3, 3)
    roof["algorithmic_bytes"] = int(alg_bytes)
    roof["algorithmic_flop"] = flop

    # ---- dense bf16 comparator --------------------------------------------------
    dense = None
    if not args.no_dense and xdt == torch.bfloat16:
        with torch.cuda.stream(stream):
            Wd = W.to(torch.bfloat16)                                  # [O, C] dense
            Bt = Wd.t().contiguous()
            if not wl.conv:
                # FC: the GEMM reads the same rotated activations as the CCI kernel
                for i in range(5):
                    torch.matmul(Xs[i % ncopy], Bt)
                gemm_ms, _ = _dense_time(lambda i: torch.matmul(Xs[i % ncopy], Bt), max(ncopy, 8), stream)
                dense = {"gemm_ms": round(gemm_ms, 5), "speedup_vs_gemm": round(gemm_ms / conv_avg, 3),
                         "note": "hipBLASLt bf16 GEMM of the dense weights, X rotated like the CCI kernel"}
            else:
                if wl.KH == 1 and wl.stride == 1 and wl.pad == 0:
                    A = Xs[0].reshape(wl.N, wl.Cin)
                else:
                    A = torch.nn.functional.unfold(Xs[0].permute(0, 3, 1, 2).float(), (wl.KH, wl.KW),
                                                   padding=wl.pad, stride=wl.stride)   # [B, Cin*k*k, L]
                    A = A.reshape(wl.B, wl.Cin, wl.KH, wl.KW, -1).permute(0, 4, 2, 3, 1).reshape(wl.N, wl.C)
                    A = A.to(torch.bfloat16).contiguous()
                Wc = W.reshape(wl.O, wl.KH, wl.KW, wl.Cin).permute(0, 3, 1, 2).to(torch.bfloat16).contiguous(
                    memory_format=torch.channels_last)
                Xn = [x.permute(0, 3, 1, 2) for x in Xs]                   # channels_last views, rotated
                for i in range(5):                                         # library heuristics / autotuning
                    torch.matmul(A, Bt)
                    torch.nn.functional.conv2d(Xn[i % ncopy], Wc, stride=wl.stride, padding=wl.pad)
                gemm_ms, _ = _dense_time(lambda i: torch.matmul(A, Bt), 8, stream)
                conv_ms_d, _ = _dense_time(lambda i: torch.nn.functional.conv2d(Xn[i % ncopy], Wc, stride=wl.stride,
                                                                               padding=wl.pad), max(ncopy, 8), stream)
                dense = {"gemm_explicit_im2col_ms": round(gemm_ms, 5), "miopen_conv2d_ms": round(conv_ms_d, 5),
                         "speedup_vs_gemm": round(gemm_ms / conv_avg, 3),
                         "speedup_vs_conv2d": round(conv_ms_d / conv_avg, 3),
                         "note": "conv2d rotates X like the CCI kernel; the GEMM reads one im2col matrix "
                                 "(warm in MALL)"}
                del A

    # ---- CPU oracle baseline (rank 0, N=1 only) ---------------------------------
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        Xf = X_cpu.float().numpy()
        t = time.perf_counter()
        v32, ix = oracle.pack(W_np, wl.G, wl.K)
        vb = oracle.bf16_bits_to_f32(oracle.bf16_rne(v32)) if vdt == torch.bfloat16 else v32
        Wm = oracle.unpack(vb, ix, wl.G).reshape(wl.O, wl.KH, wl.KW, wl.Cin)

        def oracle_rows(pix):  # the product for a sample of output pixels / rows
            if wl.conv:
                return oracle.conv2d_nhwc(Xf, Wm, stride, pad, pixels=pix)
            return oracle.spmm_rows(Xf, vb, ix, wl.G, rows=pix)

        t_pack = time.perf_counter() - t
        rng = np.random.default_rng(0)
        n = 256
        while True:
            pix = np.sort(rng.choice(wl.N, size=min(n, wl.N), replace=False))
            t = time.perf_counter()
            oracle_rows(pix)
            dt = time.perf_counter() - t
            if dt >= args.cpu_seconds or n >= wl.N:
                break
            n = min(wl.N, max(2 * n, int(n * args.cpu_seconds / max(dt, 1e-3) * 1.05)))
        reps = 1
        if len(pix) == wl.N and dt < args.cpu_seconds:
            # the whole workload fits the time budget: repeat it and keep the median
            reps = int(min(20, max(1, args.cpu_seconds // 2 / max(dt, 1e-3))))
            ts = [dt]
            for _ in range(reps - 1):
                t = time.perf_counter()
                oracle_rows(pix)
                ts.append(time.perf_counter() - t)
            dt = float(np.median(ts))
        per_pix = dt / len(pix)
        t_step = t_pack + per_pix * wl.N
        cpu_model = ""
        try:
            with open("/proc/cpuinfo") as fh:
                cpu_model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "")
        except OSError:
            pass
        cpu = {"value": round(flop / t_step / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.num_threads(),
               "kind": "oracle",
               "sample": f"oracle pack of all {wl.O}x{wl.C} weights ({t_pack:.3f}s) + the product for "
                         f"{len(pix)} of {wl.N} {'output pixels' if wl.conv else 'rows'} ({dt:.2f}s, median of {reps}, double precision), "
                         f"scaled to the full step",
               "cpu_model": cpu_model, "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}

    out = {
        "metric": "CCI-sparse GEMM effective TFLOP/s (2*N*nnz) + speedup vs dense bf16 GEMM",
        "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": (f"{wl.name}: conv {wl.KH}x{wl.KW} s{wl.stride} p{wl.pad}, batch {wl.B}, "
                                f"{wl.H}x{wl.W}, {wl.Cin}->{wl.O}, G={wl.G}, K={wl.K}, bf16 in/out, fp32 acc"
                                if wl.conv else
                                f"{wl.name}: FC, X [{wl.N},{wl.C}], W [{wl.O},{wl.C}], G={wl.G}, K={wl.K}, "
                                f"bf16 in/out, fp32 acc"),
                   "N": wl.N, "C": wl.C, "O": wl.O, "G": wl.G, "K": wl.K, "nnz": wl.nnz, "algo": algo,
                   "rotated_copies": ncopy},
        "kernels_us": {"cci_pack": round(pack_avg * 1e3, 3), kname: round(conv_avg * 1e3, 3),
                       "note": "each kernel alone, launched back to back from a HIP graph on the bench stream, "
                               "event-timed"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "dense_bf16": dense,
        "wall_s": round(wall, 3),
        "launch": "hip_graph_8_steps" if args.graph else "eager",
        "source_hash": src_hash,
    }
    print(json.dumps(out), flush=True)


def own_roof(flop, alg_bytes, t_ms, dense_flop=None):
    """Roofline of the method's own work: algorithmic bytes against HBM and
    2 * N * nnz flop against the bf16 matrix-core peak, whichever takes
    longer; `frac` = that lower bound / the measured time.  With dense_flop
    (the expanded product the matrix cores execute) the matrix-core
    utilisation on it is added as a separate figure."""
    t_hbm = alg_bytes / (PEAK["hbm_GBps"] * 1e9)
    t_mfma = flop / (PEAK["mfma_bf16_TFLOPs"] * 1e12)
    t = t_ms * 1e-3
    if t_hbm >= t_mfma:
        r = {"bound": "hbm", "achieved": round(alg_bytes / t / 1e9, 1), "peak": PEAK["hbm_GBps"], "unit": "GB/s",
             "frac": round(t_hbm / t, 4)}
    else:
        r = {"bound": "mfma", "achieved": round(flop / t / 1e12, 2), "peak": PEAK["mfma_bf16_TFLOPs"],
             "unit": "TFLOP/s", "frac": round(t_mfma / t, 4)}
    if dense_flop is not None:
        r["mfma_expanded_util"] = round(dense_flop / t / 1e12 / PEAK["mfma_bf16_TFLOPs"], 4)
    return r


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            return next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "")
    except OSError:
        return ""


def oracle_rate(wl, seconds, threads=None):
    """The oracle (pack of every weight + the product in double precision)
    timed on a bounded sample of output rows / pixels of `wl`, grown until it
    takes about `seconds`; returns (flop/s of the whole step extrapolated from
    the sample, description).  `threads` (None: all) sets the oracle's
    OpenMP threads for the measurement."""
    import numpy as np
    import oracle
    X_cpu, W_np = workloads_draw(wl)
    Xf = X_cpu.float().numpy()
    n_all = oracle.num_threads()
    if threads:
        oracle.set_num_threads(threads)
    try:
        t = time.perf_counter()
        v32, ix = oracle.pack(W_np, wl.G, wl.K)
        vb = oracle.bf16_bits_to_f32(oracle.bf16_rne(v32)) if wl.x_dtype == "bf16" else v32
        t_pack = time.perf_counter() - t
        Wm = oracle.unpack(vb, ix, wl.G).reshape(wl.O, wl.KH, wl.KW, wl.Cin) if wl.conv else None

        def rows(pix):
            if wl.conv:
                return oracle.conv2d_nhwc(Xf, Wm, (wl.stride,) * 2, (wl.pad,) * 2, pixels=pix)
            return oracle.spmm_rows(Xf, vb, ix, wl.G, rows=pix)

        rng = np.random.default_rng(0)
        n = 16
        while True:
            pix = np.sort(rng.choice(wl.N, size=min(n, wl.N), replace=False))
            t = time.perf_counter()
            rows(pix)
            dt = time.perf_counter() - t
            if dt >= seconds or n >= wl.N:
                break
            n = min(wl.N, max(2 * n, int(n * seconds / max(dt, 1e-3) * 1.05)))
        reps = 1
        if len(pix) == wl.N and dt < seconds:
            reps = int(min(20, max(1, seconds // 2 / max(dt, 1e-3))))
            ts = [dt]
            for _ in range(reps - 1):
                t = time.perf_counter()
                rows(pix)
                ts.append(time.perf_counter() - t)
            dt = float(np.median(ts))
        used = oracle.num_threads()
    finally:
        oracle.set_num_threads(n_all)
    t_step = t_pack + dt / len(pix) * wl.N
    desc = (f"{wl.name}: oracle pack of all {wl.O}x{wl.C} weights ({t_pack:.3f}s) + the product for "
            f"{len(pix)} of {wl.N} {'output pixels' if wl.conv else 'rows'} ({dt:.2f}s, median of {reps}, "
            f"double precision), scaled to the full step")
    return 2.0 * wl.N * wl.nnz / t_step, desc, used


def workloads_draw(wl):
    from paper_1910_11971_amd import workloads
    return workloads.draw(wl)


def bbs_compare(Xs, Ys, W, ncopy, stream, dense, per_k):
    """The 4096^3 FC with balanced groups (G inputs of one row, K kept) on the
    2:4 sparse matrix cores, next to the CCI product of the same (G, K), and
    the CCI layer's backward product dX = dY . W_hat through the 2:4 operand
    of W_hat^T.  Effective flop 2 * N * nnz; the sparse matrix cores execute
    half of the dense product (2 * N * M * R / 2) at twice the dense rate."""
    import torch
    from paper_1910_11971_amd import cci
    N, C = Xs[0].shape
    O = W.shape[0]
    out = {}
    x_bytes = N * C * 2
    y_bytes = N * O * 2
    for G, K in ((4, 2), (16, 1), (16, 2)):
        vals, idx = cci.bbs_pack(W, G, K)
        av, ai = cci.bbs_to_2of4(vals, idx, G)
        t_pack = _graph_time(lambda i: cci.bbs_pack(W, G, K, out=(vals, idx)), 8, 8, stream)
        t_prep = _graph_time(lambda i: cci.bbs_to_2of4(vals, idx, G), 4, 4, stream)
        t = _graph_time(lambda i: cci.spmm_2of4(Xs[i % ncopy], av, ai, out=Ys[i % ncopy]), ncopy,
                        max(2, 90 // ncopy), stream)
        nnz = O * C * K // G
        flop = 2.0 * N * nnz
        alg_bytes = x_bytes + av.numel() * 2 + ai.numel() * 2 + y_bytes   # X, the 2:4 operand, Y
        r = own_roof(flop, alg_bytes, t)
        r["smfmac_util"] = round(2.0 * N * O * C / 2 / (t * 1e-3) / 1e12 / (2 * PEAK["mfma_bf16_TFLOPs"]), 4)
        e = {"product_us": round(t * 1e3, 3), "bbs_pack_us": round(t_pack * 1e3, 3),
             "to_2of4_us": round(t_prep * 1e3, 3), "eff_TFLOPs": round(flop / (t * 1e-3) / 1e12, 2),
             "roofline": r}
        if dense:
            e["speedup_vs_dense_gemm"] = round(dense["gemm_ms"] / t, 3)
        # the CCI product of the same (G, K)
        if G == 16 and K in per_k:
            t_cci = per_k[K]["t_prod"]
        else:
            cv, ci = cci.pack(W, G, K, torch.bfloat16)
            t_cci = _graph_time(lambda i: cci.spmm(Xs[i % ncopy], cv, ci, G, out=Ys[i % ncopy]), ncopy,
                                max(2, 90 // ncopy), stream)
        e["cci_product_us"] = round(t_cci * 1e3, 3)
        e["bbs_speedup_vs_cci"] = round(t_cci / t, 3)
        # CCI backward: dX = dY . W_hat (dY shaped like Y: [N, O]) through the 2:4 operand of W_hat^T
        if O % 64 == 0:
            cv, ci = cci.pack(W, G, K, torch.bfloat16)
            tv, ti = cci.to_2of4_transposed(cv, ci, G)
            dX = [torch.empty((N, C), dtype=torch.bfloat16, device=W.device) for _ in range(2)]
            t_bwd = _graph_time(lambda i: cci.spmm_2of4(Xs[i % ncopy], tv, ti, out=dX[i % 2]), ncopy,
                                max(2, 90 // ncopy), stream)
            e["cci_backward_dX_us"] = round(t_bwd * 1e3, 3)
            if dense:
                e["cci_backward_speedup_vs_dense_gemm"] = round(dense["gemm_ms"] / t_bwd, 3)
            del tv, ti, dX
        out[f"G{G}_K{K}"] = e
        del vals, idx, av, ai
    out["note"] = ("balanced groups: G inputs of one output row keep K (Sec. 2.4, 3.3); run as a 2:4 operand "
                   "(2 values + 2-bit positions per 4 inputs) on v_smfmac_f32_16x16x64_bf16; cci_backward_dX: "
                   "dX = dY . W_hat of the CCI layer with the same (G, K), dY = the rotated X")
    return out


def td_compare(Xs, W, ncopy, stream, per_k):
    """Kernels of an improved-targeted-dropout step on the 4096^3 layer (G = 16):
    the candidate-dropout mask (HBM-bound: W and 32-bit random words read, W_eff
    bf16 and the keep mask written), and once the mask is fixed the gradient of
    the packed values (bf16: the dense dY^T X tiles on the matrix cores, kept
    entries written) next to the dense weight gradient dY^T X on hipBLASLt.
    dY is the rotated X."""
    import torch
    from paper_1910_11971_amd import cci
    N, C = Xs[0].shape
    O = W.shape[0]
    G = 16
    bits = torch.randint(-2**31, 2**31 - 1, (O, C), dtype=torch.int32, device=W.device)
    We = torch.empty((O, C), dtype=torch.bfloat16, device=W.device)
    keep = torch.empty((O, C), dtype=torch.uint8, device=W.device)
    n_t, p = cci.td_schedule(3, 4, G, 4)
    t_mask = _graph_time(lambda i: cci.td_mask(W, G, n_t, bits, p, out=(We, keep)), 4, 8, stream)
    mask_bytes = O * C * (4 + 4 + 2 + 1)
    out = {"td_mask_us": round(t_mask * 1e3, 3), "td_mask": {"n_target": n_t, "drop_rate": p},
           "td_mask_roofline": own_roof(0.0, mask_bytes, t_mask)}
    dYt = Xs[1 % ncopy].t().contiguous()
    dW = torch.empty((O, C), dtype=torch.bfloat16, device=W.device)
    t_dw, how = _dense_time(lambda i: torch.matmul(dYt, Xs[i % ncopy], out=dW), 4, stream)
    out["dense_dW_gemm_us"] = round(t_dw * 1e3, 3)
    out["dense_timing"] = how
    for K in (1, 2, 4):
        idx = per_k[K]["idx"]
        dv = torch.empty(tuple(idx.shape), dtype=torch.float32, device=W.device)
        t = _graph_time(lambda i: cci.grad_packed(Xs[(i + 1) % ncopy], Xs[i % ncopy], idx, G, out=dv), 4, 4, stream)
        nnz = O * C * K // G
        flop = 2.0 * N * nnz
        alg_bytes = 2 * N * O + 2 * N * C + nnz * 5
        out[f"grad_packed_K{K}"] = {"us": round(t * 1e3, 3), "eff_TFLOPs": round(flop / (t * 1e-3) / 1e12, 2),
                                    "kernel": "cci_grad_mfma",
                                    "roofline": own_roof(flop, alg_bytes, t, dense_flop=2.0 * N * O * C),
                                    "speedup_vs_dense_dW": round(t_dw / t, 3)}
    out["note"] = ("re-projection = cci_pack (sweep_k pack_us); backward dX of the fixed-mask layer = "
                   "bbs_2of4 cci_backward_dX_us")
    return out


def smalln_compare(Xs, W, stream, with_dense):
    """Few-row products of the 4096 x 4096 layer (G = 16) where the packed
    weight bytes set the time: cci_spmm_bits with 4-bit (log2 G) indices
    against the same kernel reading the byte indices, the library's choice
    (cci_spmm) and a dense bf16 GEMM of the same shape.  Roofline: HBM on
    X + packed values + indices + Y, with each launch reading fresh weights
    (8 packed copies rotated)."""
    import torch
    from paper_1910_11971_amd import cci
    C = Xs[0].shape[1]
    O = W.shape[0]
    G = 16
    b = cci.index_width(G)
    out = {}
    Wd_t = W.to(torch.bfloat16).t().contiguous()
    copies = 8
    for K in (1, 4):
        packs = [cci.pack(W * (1.0 + 0.001 * i), G, K, torch.bfloat16) for i in range(copies)]
        streams = [cci.index_bits(ix, b) for _, ix in packs]
        nnz = O * C * K // G
        for N in (1, 16, 64):
            X = Xs[0][:N].contiguous()
            Y = torch.empty((N, O), dtype=torch.bfloat16, device=W.device)
            t_bits = _graph_time(lambda i: cci.spmm_bits(X, packs[i % copies][0], streams[i % copies], G, b, out=Y),
                                 copies, 8, stream)
            t_byte = _graph_time(lambda i: cci.spmm_bits(X, packs[i % copies][0], packs[i % copies][1], G, 8, out=Y),
                                 copies, 8, stream)
            t_auto = _graph_time(lambda i: cci.spmm(X, packs[i % copies][0], packs[i % copies][1], G, out=Y),
                                 copies, 8, stream)
            flop = 2.0 * N * nnz
            io = N * C * 2 + N * O * 2
            bytes_bits = io + nnz * 2 + (nnz * b + 7) // 8
            bytes_byte = io + nnz * 3
            e = {"bits_us": round(t_bits * 1e3, 3), "bytes_us": round(t_byte * 1e3, 3),
                 "auto_us": round(t_auto * 1e3, 3),
                 "bits_roofline": own_roof(flop, bytes_bits, t_bits),
                 "bytes_roofline": own_roof(flop, bytes_byte, t_byte),
                 "alg_bytes_bits": bytes_bits, "alg_bytes_uint8": bytes_byte}
            if with_dense:
                t_d = _graph_time(lambda i: torch.matmul(X, Wd_t, out=Y), copies, 8, stream)
                e["dense_gemm_us"] = round(t_d * 1e3, 3)
                e["speedup_bits_vs_dense"] = round(t_d / t_bits, 3)
            out[f"K{K}_N{N}"] = e
        del packs, streams
    out["note"] = (f"index width {b} bits (ceil(log2 16)) vs 8; the dense GEMM reads one 32 MB weight copy "
                   "(warm in the last-level cache), the CCI kernels rotate 8 packed copies")
    return out


def main_fc_sweep(args):
    """The 4096^3 FC layer, G = 16: the timed steps at K = args.k, and every K
    of the sweep measured kernel by kernel in the same process."""
    import numpy as np
    import torch
    from paper_1910_11971_amd import cci, workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream(device=dev)  # default priority
    Ks = (1, 2, 4, 8, 16)
    if args.k not in Ks:
        raise SystemExit(f"--k must be one of {Ks}")
    wl0 = workloads.WORKLOADS["fc4096_k1"]
    X_cpu, W_np = workloads.draw(wl0)       # X and W do not depend on K (same seed, same draws)
    x_bytes = X_cpu.numel() * 2
    y_bytes = wl0.N * wl0.O * 2
    ncopy = 1 if args.rotate_mb <= 0 else max(1, int(np.ceil(args.rotate_mb * 1e6 / (x_bytes + y_bytes))))
    X0 = X_cpu.to(dev)
    Xs = [X0] + [X0.clone() for _ in range(ncopy - 1)]
    Ys = [torch.empty((wl0.N, wl0.O), dtype=torch.bfloat16, device=dev) for _ in range(ncopy)]
    W = torch.from_numpy(W_np).to(dev)
    Wd_t = W.to(torch.bfloat16).t().contiguous()      # dense comparator's B operand [C, O]

    per_k = {}
    for K in Ks:
        wl = workloads.WORKLOADS[f"fc4096_k{K}"]
        vals = torch.empty((wl.O // wl.G, K, wl.C), dtype=torch.bfloat16, device=dev)
        idx = torch.empty((wl.O // wl.G, K, wl.C), dtype=torch.uint8, device=dev)
        with torch.cuda.stream(stream):
            cci.pack(W, wl.G, K, torch.bfloat16, out=(vals, idx))
        algo = cci.auto_algo(torch.bfloat16, torch.bfloat16, wl.N, wl.C, wl.Cin, wl.O, wl.G, K)
        prod = (lambda i, vals=vals, idx=idx, G=wl.G: cci.spmm(Xs[i % ncopy], vals, idx, G,
                                                               out_dtype=torch.bfloat16, out=Ys[i % ncopy]))
        pack = (lambda i, vals=vals, idx=idx, G=wl.G, K=K: cci.pack(W, G, K, torch.bfloat16, out=(vals, idx)))
        t_prod = _graph_time(prod, ncopy, max(2, 90 // ncopy), stream)
        t_pack = _graph_time(pack, 8, 8, stream)
        flop = 2.0 * wl.N * wl.nnz
        dense_flop = 2.0 * wl.N * wl.C * wl.O
        alg_bytes = x_bytes + wl.nnz * 3 + y_bytes
        per_k[K] = dict(wl=wl, vals=vals, idx=idx, algo=algo, prod=prod, pack=pack, t_prod=t_prod, t_pack=t_pack,
                        flop=flop, dense_flop=dense_flop, alg_bytes=alg_bytes)

    # dense bf16 comparator: hipBLASLt on the same rotated X, captured like the CCI kernels
    dense = None
    if not args.no_dense:
        gemm = lambda i: torch.matmul(Xs[i % ncopy], Wd_t, out=Ys[i % ncopy])
        try:
            t_gemm, how = _graph_time(gemm, ncopy, max(2, 90 // ncopy), stream), "hip_graph"
        except RuntimeError:
            t_gemm, how = _eager_time(gemm, 60, stream), "eager"
        dense = {"gemm_ms": round(t_gemm, 5), "timing": how,
                 "note": "torch.matmul bf16 (hipBLASLt, fp32 accumulate, bf16 out) of the dense weights, "
                         "X rotated like the CCI kernel"}

    # ---- balanced sparsity on the 2:4 sparse matrix cores, same shape -------------
    bbs = None if args.no_bbs else bbs_compare(Xs, Ys, W, ncopy, stream, dense, per_k)
    td = None if args.no_td else td_compare(Xs, W, ncopy, stream, per_k)
    smalln = None if args.no_smalln else smalln_compare(Xs, W, stream, dense is not None)

    # ---- timed region: whole steps (pack + product) at the declared K ------------
    sel = per_k[args.k]
    wl = sel["wl"]

    def step(i):
        sel["pack"](i)
        sel["prod"](i)

    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(args.steps):
            step(i)
        b.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    ms_step = a.elapsed_time(b) / args.steps
    value = sel["flop"] / (ms_step * 1e-3) / 1e12

    kname = kernel_name(sel["algo"])
    src_hash = kernel_source_hash(kname)
    roof = own_roof(sel["flop"], sel["alg_bytes"], sel["t_prod"], sel["dense_flop"])
    roof["traffic"] = load_traffic(wl.name, kname, src_hash)
    roof.update({"kernel": kname, "kernel_avg_us": round(sel["t_prod"] * 1e3, 3),
                 "algorithmic_bytes": int(sel["alg_bytes"]), "algorithmic_flop": sel["flop"],
                 "expanded_flop": sel["dense_flop"]})

    sweep_k = {}
    for K, d in per_k.items():
        r = own_roof(d["flop"], d["alg_bytes"], d["t_prod"], d["dense_flop"])
        e = {"algo": d["algo"], "product_us": round(d["t_prod"] * 1e3, 3), "pack_us": round(d["t_pack"] * 1e3, 3),
             "eff_TFLOPs": round(d["flop"] / (d["t_prod"] * 1e-3) / 1e12, 2),
             "roofline": {"bound": r["bound"], "frac": r["frac"], "mfma_expanded_util": r["mfma_expanded_util"]}}
        if dense:
            e["speedup_vs_dense_gemm"] = round(dense["gemm_ms"] / d["t_prod"], 3)
        sweep_k[str(K)] = e

    cpu = None
    if not args.no_cpu_baseline:
        rate, desc, used = oracle_rate(wl, args.cpu_seconds)
        cpu = {"value": round(rate / 1e12, 6), "unit": "TFLOP/s", "cores": used, "kind": "oracle", "sample": desc,
               "cpu_model": _cpu_model(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
               "nproc": os.cpu_count()}
        r1, d1, _ = oracle_rate(wl, max(1.0, args.cpu_seconds / 4), threads=1)
        cpu["one_core"] = {"value": round(r1 / 1e12, 7), "unit": "TFLOP/s", "sample": d1}
        if not args.no_cpu_configs:
            cfgs = {}
            for name in ("fc256", "conv3x3", "conv1x1_k4", "conv1x1_k2"):
                w = workloads.WORKLOADS[name]
                ra, _, ua = oracle_rate(w, 1.5)
                r1, _, _ = oracle_rate(w, 1.5, threads=1)
                cfgs[name] = {"all_cores_TFLOPs": round(ra / 1e12, 7), "cores": ua,
                              "one_core_TFLOPs": round(r1 / 1e12, 7)}
            cpu["configs"] = cfgs

    out = {
        "metric": "CCI-sparse GEMM effective TFLOP/s (2*N*nnz) + speedup vs dense bf16 GEMM",
        "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": (f"{wl.name}: sparsity-sweep FC, X bf16 [4096,4096] ~N(0,1), W [4096,4096] "
                                f"~N(0,1/4096), G=16, K={args.k} ({100 * (1 - args.k / 16):.2f}% sparse), fp32 acc, "
                                f"bf16 out; step = cci_pack + cci_spmm; every K of the sweep under sweep_k"),
                   "N": wl.N, "C": wl.C, "O": wl.O, "G": wl.G, "K": wl.K, "nnz": wl.nnz, "algo": sel["algo"],
                   "rotated_copies": ncopy},
        "kernels_us": {"cci_pack": round(sel["t_pack"] * 1e3, 3), kname: round(sel["t_prod"] * 1e3, 3),
                       "note": "each kernel alone, launched back to back from a HIP graph on the bench stream, "
                               "event-timed"},
        "roofline": roof,
        "sweep_k": sweep_k,
        "bbs_2of4": bbs,
        "td_step": td,
        "few_rows_bits": smalln,
        "cpu_baseline": cpu,
        "dense_bf16": dense,
        "speedup_vs_dense_gemm": None if dense is None else round(dense["gemm_ms"] / sel["t_prod"], 3),
        "wall_s": round(wall, 3),
        "launch": "eager",
        "source_hash": src_hash,
    }
    print(json.dumps(out), flush=True)


def _graph_time(fn, n_launch, reps, stream):
    """Average duration of fn(i) for i < n_launch, captured in one HIP graph
    and replayed `reps` times (no host launch cost between kernels)."""
    import torch
    with torch.cuda.stream(stream):
        for i in range(n_launch):
            fn(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for i in range(n_launch):
            fn(i)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        g.replay()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(reps):
            g.replay()
        b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (reps * n_launch)


def _eager_time(fn, n, stream):
    import torch
    with torch.cuda.stream(stream):
        for i in range(5):
            fn(i)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(n):
            fn(i)
        b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n


def kernel_name(algo):
    return {"dense_tile_mfma": "cci_dense_tile", "wide_tile_mfma": "cci_wide_tile",
            "narrow_mfma": "cci_narrow", "resident_mfma": "cci_resident",
            "few_rows_mfma": "cci_bits", "tap_tile_mfma": "cci_tap_tile",
            "stream_tile_mfma": "cci_stream_tile", "split_k_mfma": "cci_split_k"}.get(algo, "cci_sparse_mac")


def _dense_time(fn, n_launch, stream, reps=10):
    """A dense comparator timed like the CCI kernels (HIP-graph replays of
    n_launch calls); eager launches if the library call cannot be captured.
    Returns (ms per call, "hip_graph" | "eager")."""
    try:
        return _graph_time(fn, n_launch, reps, stream), "hip_graph"
    except RuntimeError:
        import torch
        torch.cuda.synchronize()
        return _eager_time(fn, max(10, n_launch * reps // 2), stream), "eager"


def roof_for(kname, flop, dense_flop, alg_bytes, t_ms):
    """The matrix-core kernels against the method's own work (own_roof); the
    vector-ALU kernel multiplies only kept weights, so its bound is the fp32
    FMA rate (or HBM, if that takes longer)."""
    if kname in ("cci_dense_tile", "cci_wide_tile", "cci_narrow", "cci_resident", "cci_bits", "cci_tap_tile",
                 "cci_stream_tile", "cci_split_k"):
        return own_roof(flop, alg_bytes, t_ms, dense_flop)
    t_alu = flop / (PEAK["valu_fp32_TFLOPs"] * 1e12)
    t_hbm = alg_bytes / (PEAK["hbm_GBps"] * 1e9)
    t = t_ms * 1e-3
    if t_hbm > t_alu:
        return {"bound": "hbm", "achieved": round(alg_bytes / t / 1e9, 1), "peak": PEAK["hbm_GBps"],
                "unit": "GB/s", "frac": round(t_hbm / t, 4)}
    return {"bound": "alu", "achieved": round(flop / t / 1e12, 2), "peak": PEAK["valu_fp32_TFLOPs"],
            "unit": "TFLOP/s", "frac": round(t_alu / t, 4)}


def sweep(args):
    """One JSON line per configuration: CCI kernel time (HIP-graph replays over
    rotated inputs), cci_pack time, effective TFLOP/s (2*N*nnz), the roofline
    fraction, and the dense bf16 comparators of the same shape."""
    import numpy as np
    import torch
    from paper_1910_11971_amd import cci, workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream(device=dev)
    names = ["fc256", "conv3x3", "conv1x1_k4", "conv1x1_k2"] + [f"fc4096_k{k}" for k in (1, 2, 4, 8, 16)]
    only = set(x for x in args.sweep_only.split(",") if x)
    if only:
        names = [n for n in names if n in only]
    for name in names:
        wl = workloads.WORKLOADS[name]
        X_cpu, W_np = workloads.draw(wl)
        xdt = torch.bfloat16 if wl.x_dtype == "bf16" else torch.float32
        ydt = torch.bfloat16 if wl.y_dtype == "bf16" else torch.float32
        ysz = 2 if ydt == torch.bfloat16 else 4
        x_bytes = X_cpu.numel() * X_cpu.element_size()
        y_bytes = wl.N * wl.O * ysz
        ncopy = max(1, int(np.ceil(args.rotate_mb * 1e6 / (x_bytes + y_bytes)))) if args.rotate_mb > 0 else 1
        ncopy = min(ncopy, 24)
        Xs = [X_cpu.to(dev) for _ in range(ncopy)]
        if wl.conv:
            Ys = [torch.empty((wl.B, wl.Ho, wl.Wo, wl.O), dtype=ydt, device=dev) for _ in range(ncopy)]
        else:
            Ys = [torch.empty((wl.N, wl.O), dtype=ydt, device=dev) for _ in range(ncopy)]
        W = torch.from_numpy(W_np).to(dev)
        vals, idx = cci.pack(W, wl.G, wl.K, xdt)
        algo = cci.auto_algo(xdt, xdt, wl.N, wl.C, wl.Cin, wl.O, wl.G, wl.K)
        kname = kernel_name(algo)
        if wl.conv:
            f = lambda i: cci.conv_im2col(Xs[i % ncopy], vals, idx, wl.G, wl.KH, wl.KW, (wl.stride,) * 2,
                                          (wl.pad,) * 2, out_dtype=ydt, out=Ys[i % ncopy])
        else:
            f = lambda i: cci.spmm(Xs[i % ncopy], vals, idx, wl.G, out_dtype=ydt, out=Ys[i % ncopy])
        n_launch = max(ncopy, 8)
        t_cci = _graph_time(f, n_launch, max(2, 200 // n_launch), stream)
        t_pack = _graph_time(lambda i: cci.pack(W, wl.G, wl.K, xdt, out=(vals, idx)), 16, 10, stream)
        flop = 2.0 * wl.N * wl.nnz
        dense_flop = 2.0 * wl.N * wl.C * wl.O
        alg_bytes = x_bytes + wl.nnz * ((2 if xdt == torch.bfloat16 else 4) + 1) + y_bytes
        out = {"workload": name, "N": wl.N, "C": wl.C, "O": wl.O, "G": wl.G, "K": wl.K, "algo": algo,
               "cci_ms": round(t_cci, 5), "pack_ms": round(t_pack, 5),
               "eff_TFLOPs": round(flop / (t_cci * 1e-3) / 1e12, 3),
               "roofline": roof_for(kname, flop, dense_flop, alg_bytes, t_cci), "rotated_copies": ncopy}
        if xdt == torch.bfloat16:
            Wd = W.to(torch.bfloat16)
            Bt = Wd.t().contiguous()
            if wl.conv and not (wl.KH == 1 and wl.stride == 1 and wl.pad == 0):
                A = torch.nn.functional.unfold(Xs[0].permute(0, 3, 1, 2).float(), (wl.KH, wl.KW), padding=wl.pad,
                                               stride=wl.stride)
                A = A.reshape(wl.B, wl.Cin, wl.KH, wl.KW, -1).permute(0, 4, 2, 3, 1).reshape(wl.N, wl.C)
                As = [A.to(torch.bfloat16).contiguous()]
                del A
            else:
                As = [x.reshape(wl.N, wl.C) for x in Xs]
            t_gemm, how = _dense_time(lambda i: torch.matmul(As[i % len(As)], Bt), max(len(As), 8), stream)
            out["dense_gemm_ms"] = round(t_gemm, 5)
            out["dense_timing"] = how
            out["speedup_vs_dense_gemm"] = round(t_gemm / t_cci, 3)
            if wl.conv:
                Wc = W.reshape(wl.O, wl.KH, wl.KW, wl.Cin).permute(0, 3, 1, 2).to(torch.bfloat16).contiguous(
                    memory_format=torch.channels_last)
                Xn = [x.permute(0, 3, 1, 2) for x in Xs]
                t_conv, _ = _dense_time(lambda i: torch.nn.functional.conv2d(Xn[i % ncopy], Wc, stride=wl.stride,
                                                                             padding=wl.pad), max(ncopy, 8), stream)
                out["miopen_conv2d_ms"] = round(t_conv, 5)
                out["speedup_vs_conv2d"] = round(t_conv / t_cci, 3)
            del As
        print(json.dumps(out), flush=True)
        del Xs, Ys, W, vals, idx
        torch.cuda.empty_cache()
    if not only or "resnet50" in only:
        sweep_resnet50(stream)
    if not only or "mobilenetv2" in only:
        for K in (int(k) for k in args.mbv2_k.split(",")):
            sweep_mobilenetv2(stream, K)


def sweep_resnet50(stream):
    """ResNet-50-shaped forward at batch 64: the CCI network (one HIP graph per
    forward) against the same network with dense bf16 weights on torch's
    channels-last convolutions."""
    import numpy as np
    import torch
    from paper_1910_11971_amd import workloads
    from paper_1910_11971_amd.resnet import ResNet50CCI

    net = workloads.ResNet50()
    X, ws, fcw = workloads.draw_resnet50(net)
    dev = torch.device("cuda:0")
    model = ResNet50CCI(net, ws, fcw, device=dev)
    Xd = X.to(dev)
    t_cci = _graph_time(lambda i: model.forward(Xd), 1, 10, stream)
    # effective flop of the CCI network: 2 * N * nnz summed over its layers
    flop = 0.0
    rec = []
    model.forward(Xd, record=rec)
    torch.cuda.synchronize()
    for kind, key, inp, out, res in rec:
        if kind == "conv":
            L = net.layers[key]
            flop += 2.0 * (out.numel() // L.Cout) * L.Cout * L.fan_in * L.K / net.G
        elif kind == "fc":
            flop += 2.0 * out.shape[0] * out.shape[1] * inp.shape[1]
    del rec
    # dense bf16 reference network, same layer sequence
    sc = 1.0 / np.sqrt(1.0 + workloads.BN_EPS)  # batch norm at its initial state, folded into the weights
    Wd = [(torch.from_numpy(w).to(dev) * sc).reshape(L.Cout, L.k, L.k, L.Cin).permute(0, 3, 1, 2)
          .to(torch.bfloat16).contiguous(memory_format=torch.channels_last) for L, w in zip(net.layers, ws)]
    Wfc = torch.from_numpy(fcw).to(dev).to(torch.bfloat16)
    Xn = Xd.permute(0, 3, 1, 2)
    F = torch.nn.functional

    def dense_forward(_i):
        def cv(i, x):
            L = net.layers[i]
            return F.conv2d(x, Wd[i], stride=L.stride, padding=L.pad)
        x = F.relu(cv(0, Xn))
        x = F.max_pool2d(x, 3, 2, 1)
        i = 1
        while i < len(net.layers):
            ds = i + 3 < len(net.layers) and net.layers[i + 3].name.endswith(".ds")
            y = F.relu(cv(i, x))
            y = F.relu(cv(i + 1, y))
            ident = cv(i + 3, x) if ds else x
            x = F.relu(cv(i + 2, y) + ident)
            i += 4 if ds else 3
        p = x.float().mean(dim=(2, 3)).to(torch.bfloat16)
        return torch.matmul(p, Wfc.t().contiguous()).float()

    t_dense, how = _dense_time(dense_forward, 1, stream, reps=5)
    print(json.dumps({"workload": "resnet50", "B": net.B, "HW": net.HW, "G": net.G, "K": net.K, "dense_timing": how,
                      "cci_forward_ms": round(t_cci, 4), "eff_TFLOPs": round(flop / (t_cci * 1e-3) / 1e12, 3),
                      "dense_bf16_forward_ms": round(t_dense, 4),
                      "speedup_vs_dense": round(t_dense / t_cci, 3),
                      "images_per_s": round(net.B / (t_cci * 1e-3), 1)}), flush=True)


def sweep_mobilenetv2(stream, K, B=64):
    """The 32 CCI pointwise layers of MobileNetV2 (G = 8, s = K) at batch 64,
    each on its own synthetic input, run back to back from one HIP graph,
    against the same 32 products as dense bf16 GEMMs (hipBLASLt).  The
    layers' operands total about 1 GB, so a replay finds little of a layer in
    the caches.  Batch norm is folded into the epilogue's scale / bias, with
    ReLU after the expanding layers (the network's ReLU6 clamp at 6 is not
    part of the product).  Per-layer times come from graphs of 8 launches of
    one layer."""
    import numpy as np
    import torch
    from paper_1910_11971_amd import cci, workloads

    dev = torch.device("cuda:0")
    P = workloads.mobilenetv2_pointwise(B=B, K=K)
    kinds = [l.kind for l in workloads.mobilenetv2_cci_layers()]
    Xs, Ys, packs, Wd, As, eps = [], [], [], [], [], []
    flop = dense_flop = alg_bytes = 0.0
    for w in P:
        X_cpu, W_np = workloads.draw(w)
        Xs.append(X_cpu.to(dev))
        Ys.append(torch.empty((w.B, w.Ho, w.Wo, w.O), dtype=torch.bfloat16, device=dev))
        W = torch.from_numpy(W_np).to(dev)
        packs.append(cci.pack(W, w.G, w.K, torch.bfloat16))
        Wd.append(W.to(torch.bfloat16).t().contiguous())
        As.append(Xs[-1].reshape(w.N, w.C))
        sc, bi = workloads.bn_fold(w.O)  # batch norm folded into the epilogue
        eps.append((torch.from_numpy(sc).to(dev), torch.from_numpy(bi).to(dev)))
        flop += 2.0 * w.N * w.nnz
        dense_flop += 2.0 * w.N * w.C * w.O
        alg_bytes += 2.0 * w.N * (w.C + w.O) + 3.0 * w.nnz
    algos = [cci.auto_algo(torch.bfloat16, torch.bfloat16, w.N, w.C, w.Cin, w.O, w.G, w.K) for w in P]

    def layer(i, algo="auto"):
        w = P[i]
        vals, idx = packs[i]
        cci.conv_im2col(Xs[i], vals, idx, w.G, 1, 1, (1, 1), (0, 0), scale=eps[i][0], bias=eps[i][1],
                        relu=kinds[i] == "expand", out_dtype=torch.bfloat16, out=Ys[i], algo=algo)

    def network(_i):
        for i in range(len(P)):
            layer(i)

    def dense(_i):
        for i in range(len(P)):
            torch.matmul(As[i], Wd[i])

    t_cci = _graph_time(network, 1, 20, stream)
    t_dense, dense_how = _dense_time(dense, 1, stream, reps=20)
    per_layer = []
    for i, w in enumerate(P):
        t = _graph_time(lambda _j, i=i: layer(i), 8, 5, stream)
        row = [w.name[5:], w.N, w.C, w.O, algos[i], round(t * 1e3, 2)]
        alt = {}
        for a in ("narrow_mfma", "dense_tile_mfma"):  # the other MFMA kernels that take the shape
            if a == algos[i]:
                continue
            try:
                alt[a] = round(_graph_time(lambda _j, i=i, a=a: layer(i, a), 8, 5, stream) * 1e3, 2)
            except cci.CCIError:
                pass
        per_layer.append(row + [alt])
    t_hbm = alg_bytes / (PEAK["hbm_GBps"] * 1e9)
    print(json.dumps({"workload": f"mobilenetv2_pw_k{K}", "B": B, "G": 8, "K": K, "layers": len(P),
                      "cci_ms": round(t_cci, 4), "eff_TFLOPs": round(flop / (t_cci * 1e-3) / 1e12, 3),
                      "alg_bytes_MB": round(alg_bytes / 1e6, 1),
                      "roofline": {"bound": "hbm", "frac": round(t_hbm / (t_cci * 1e-3), 4)},
                      "dense_gemm_ms": round(t_dense, 4), "dense_timing": dense_how,
                      "speedup_vs_dense_gemm": round(t_dense / t_cci, 3),
                      "algos": {a: algos.count(a) for a in sorted(set(algos))},
                      "per_layer_us": per_layer}), flush=True)
    del Xs, Ys, packs, Wd, As, eps
    torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
