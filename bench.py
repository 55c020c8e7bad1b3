"""Throughput of the Direct-P full-MXFP4 attention forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

A step is one forward pass (QK on scaled FP4 matrix cores, Direct-P, PV, the
epilogue) over the whole workload with MXFP4 operands already resident in HBM;
the paper times the attention kernel on prequantized operands and excludes
quantization (its Sec. "Timed scope and operand contract").  The quantizer is
timed separately and reported in the same line.  The metric is the paper's
ops count 4 B H N^2 d per step (eq. hao-flops) over the step time.

Prints one JSON line.  Also reported: the same-design BF16 kernel on the same
inputs (windows interleaved with the FP4 ones, the paper's speedup
t_BF16 / t_FP4), the roofline of the forward kernel against the dense MXFP4
matrix peak (and, beside it, the shader clock the kernel ran at and the rate
a stream of FP4 matrix products alone sustains on the workload's K and Q
codes), both kernels on the shapes the paper reports (D128 and D64) next to
the paper's printed rates, and the CPU oracle timed on a
bounded sample of rows.  The
defaults follow the paper's timing protocol (Sec. "Operator benchmark suites"): 240
warmup steps (over 300 ms), 2200 timed steps (about 3 s), and ten interleaved
300 ms windows of each of the FP4 and BF16 kernels.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
MXFP4_PEAK_TFLOPS = 10100.0   # MI355X dense FP4/FP6 matrix peak
BF16_PEAK_TFLOPS = 2500.0     # MI355X dense BF16 matrix peak
HBM_PEAK_GBS = 8000.0
SPEC_CLOCK_GHZ = 2.4          # the clock the spec peaks assume
EX2_SWEEP = (1, 2, 4, 16)
GUARD_ML = (110, 16)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fwd_mxfp4_long_b1h32_n16384_d128_traffic.json")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_04105_amd", "csrc", f)
                  for f in ("fwd_mxfp4.hpp", "fwd_mxfp4.hip", "gfx950.hpp", "launch.hpp")]


def _source_sha():
    """Hash of the forward kernel's sources with comments and blank lines removed,
    so that the committed counters stay attached to the code they measured."""
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path) as f:
            for line in f:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()


def _traffic():
    """HBM bytes per forward launch from committed rocprofv3 counters, if they
    were taken on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_sha256") != _source_sha():
        return None
    return t.get("bytes_per_launch")


def traffic_summary(fetch_csv, write_csv, out_path=TRAFFIC_FILE):
    """Write the per-launch HBM traffic file from the counter CSVs of two
    ``--traffic-run`` passes (FETCH_SIZE, then WRITE_SIZE, in KiB per dispatch).
    Each counter is scaled by what it reads for the 256 MiB device copy."""
    import csv

    def per_kernel(path, counter):
        vals = {}
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] == counter:
                    vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return vals

    fetch, write = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")

    def pick(vals, key):
        hits = [v for k, v in vals.items() if key in k]
        if len(hits) != 1 or len(hits[0]) != 1:
            raise SystemExit(f"expected exactly one dispatch of {key!r} in the counter file, got {hits}")
        return hits[0][0]

    kname = "fwd_mxfp4_kernel<128, 8, false, 0, 0>"
    copy_bytes = 256 << 20
    fs = copy_bytes / 1024 / pick(fetch, "copyBuffer")
    ws = copy_bytes / 1024 / pick(write, "copyBuffer")
    fk, wk = pick(fetch, kname), pick(write, kname)
    import workloads
    w = workloads.WORKLOADS[workloads.BENCH_WORKLOAD]
    algo = w.B * w.H * (3 * w.N * w.d * (0.5 + 1 / 32) + 4 * w.N * w.d)
    res = {
        "kernel": kname,
        "workload": w.name,
        "source_sha256": _source_sha(),
        "fetch_size_kib": fk,
        "write_size_kib": wk,
        "copy_calibration": {"bytes": copy_bytes, "fetch_size_kib": pick(fetch, "copyBuffer"),
                             "write_size_kib": pick(write, "copyBuffer"), "fetch_scale": fs, "write_scale": ws},
        "fetch_bytes": fk * 1024 * fs,
        "write_bytes": wk * 1024 * ws,
        "bytes_per_launch": fk * 1024 * fs + wk * 1024 * ws,
        "algorithmic_bytes": int(algo),
        "commands": [
            "rocprofv3 --pmc FETCH_SIZE --output-format csv -d <fetch> -o fetch -- python bench.py --traffic-run",
            "rocprofv3 --pmc WRITE_SIZE --output-format csv -d <write> -o write -- python bench.py --traffic-run",
            "python bench.py --traffic-summary <fetch>/fetch_counter_collection.csv "
            "<write>/write_counter_collection.csv",
        ],
    }
    with open(out_path, "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res))


def _time_windows(torch, fns, window_ms, windows):
    """Median per-call ms of each fn over ``windows`` interleaved windows of about
    ``window_ms`` each (calls per window from a one-call estimate), timed with events
    on the current stream (the stream the kernels are launched on)."""
    calls = {}
    for name, fn in fns.items():
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record()
        fn()
        end.record()
        torch.cuda.synchronize()
        calls[name] = max(1, int(round(window_ms / max(start.elapsed_time(end), 1e-3))))
    res = {k: [] for k in fns}
    for _ in range(windows):
        for name, fn in fns.items():
            steps = calls[name]
            start = torch.cuda.Event(enable_timing=True)
            end = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            start.record()
            for _ in range(steps):
                fn()
            end.record()
            torch.cuda.synchronize()
            res[name].append(start.elapsed_time(end) / steps)
    return {k: sorted(v)[len(v) // 2] for k, v in res.items()}, res


def measured_clock_ghz(torch, fa, ops, w, launches=5):
    """Shader clock achieved by the timed forward kernel: launched through the
    test entry point with no rows to dump (the plain forward kernel), each
    workgroup records the shader-clock cycles and 100 MHz constant-clock ticks
    of its residency; the ratio of the sums over workgroups and launches."""
    no_rows = torch.zeros(0, dtype=torch.int64, device=ops[0].device)
    cyc = ticks = 0
    for _ in range(launches):
        r = fa.debug_directp_mxfp4(*ops, no_rows, softmax_scale=w.softmax_scale, wg_clock=True)
        c = r["wg_clock"].cpu()
        cyc += int(c[:, 0].sum())
        ticks += int(c[:, 1].sum())
    return cyc / (ticks / 100e6) / 1e9


def sustained_mfma_tflops(torch, fa, a_codes, b_codes, blocks=1024, iters=100000, launches=7):
    """Rate of a stream of FP4 32x32x64 matrix products with nothing else running,
    on operand bytes of the workload (the QK product's K and Q codes): the matrix
    unit's sustained ceiling on this board for this data, beside the spec peak.
    Median over ``launches`` after one warmup launch."""
    times = []
    for i in range(launches + 1):
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        _, flop = fa.debug_mfma_stream(a_codes, b_codes, blocks, iters)
        end.record()
        torch.cuda.synchronize()
        if i:
            times.append(start.elapsed_time(end))
    ms = sorted(times)[len(times) // 2]
    return flop / (ms * 1e-3) / 1e12


# The paper's retained route (NV/MX) on the shapes it reports, B1: TFLOP/s as
# printed for its GB200 and B300 systems (None: not run) -- D128 from its primary
# forward comparison (Table primary-results), D64 from its B300 D64 diagnostics
# (Table b300-d64-diagnostic).  Context for the same shapes here, not a target:
# other hardware, and NVFP4 Q/K where this path uses MXFP4.
PAPER_SHAPES = {(128, 24, 4096): (2237, 2369), (128, 64, 4096): (2711, 2901), (128, 64, 6144): (2731, 2958),
                (128, 64, 8192): (2900, 3116), (128, 64, 9472): (None, 3159), (128, 24, 32768): (2998, 2945),
                (64, 12, 4096): (None, 775), (64, 24, 4096): (None, 1105), (64, 24, 32768): (None, 1434),
                (64, 32, 2048): (None, 862), (64, 32, 32768): (None, 1438), (64, 64, 1024): (None, 672),
                (64, 64, 4096): (None, 1323), (64, 64, 32768): (None, 1439)}


def paper_shape_sweep(torch, fa, seed=20):
    """The MXFP4 forward and the BF16 kernel on the paper's reported shapes: N(0, 1)
    bf16 inputs drawn on the GPU, windows of the two kernels interleaved."""
    res = []
    g = torch.Generator(device="cuda").manual_seed(seed)
    for (d, H, S), (gb200, b300) in PAPER_SHAPES.items():
        q, k, v = (torch.randn((1, H, S, d), device="cuda", generator=g, dtype=torch.float32).to(torch.bfloat16)
                   for _ in range(3))
        ops = fa.quantize_qkv(q, k, v)
        vt = fa.transpose_bf16(v)
        out = torch.empty((1, H, S, d), dtype=torch.float32, device="cuda")
        scale = 1.0 / math.sqrt(d)
        fns = {"fp4": lambda: fa.forward_mxfp4(*ops, softmax_scale=scale, out=out),
               "bf16": lambda: fa.forward_bf16(q, k, vt, softmax_scale=scale, out=out)}
        for fn in fns.values():
            fn()
        med = _time_windows(torch, fns, 100.0, 3)[0]
        flop = 4.0 * H * S * S * d
        res.append({"shape": f"B1/S{S}/H{H}/D{d}", "tflops": round(flop / (med["fp4"] * 1e-3) / 1e12, 1),
                    "bf16_tflops": round(flop / (med["bf16"] * 1e-3) / 1e12, 1),
                    "speedup_vs_bf16": round(med["bf16"] / med["fp4"], 3),
                    "paper_nvmx_tflops": {"gb200": gb200, "b300": b300}})
        del q, k, v, ops, vt, out
    return res


def cpu_oracle_baseline(w, q, k, v, budget_s=12.0):
    """Time the oracle (as it stands) on consecutive rows of head (0, 0) of the bench
    inputs (CPU tensors q, k, v [B, H, N, d]) until the budget is spent.  Returns the
    record and the oracle's output rows, for the parity check."""
    import numpy as np
    import workloads
    from oracle import directp, mxfp4
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing: report the affinity set
        threads = len(os.sched_getaffinity(0))
    q64, k64, v64 = (workloads.as_f64(t[:1, :1])[0, 0] for t in (q, k, v))
    t0 = time.perf_counter()
    kc, ks = mxfp4.quantize(k64, axis=-1)
    vc, vs = mxfp4.quantize(v64, axis=-2)
    rows_done = 0
    chunk = 128
    outs = []
    while rows_done < w.N and time.perf_counter() - t0 < budget_s:
        qc, qs = mxfp4.quantize(q64[rows_done:rows_done + chunk], axis=-1)
        outs.append(directp.forward_rows(qc, qs, kc, ks, vc, vs, np.arange(chunk), w.softmax_scale,
                                         want_codes=False)["O"])
        rows_done += chunk
    dt = time.perf_counter() - t0
    flops = 4.0 * rows_done * w.N * w.d
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"{rows_done} query rows of head (b0,h0) of {w.name} (all {w.N} keys), "
                  f"including the oracle's own MXFP4 quantization of that head's K and V; {dt:.1f} s",
        "seconds": round(dt, 2),
        "full_workload_estimate_s": round(dt * w.rows / rows_done, 1),
    }, np.concatenate(outs)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    # defaults follow the paper's protocol: >= 300 ms of warmup, >= 3 s measured
    ap.add_argument("--steps", type=int, default=2200)
    ap.add_argument("--warmup", type=int, default=240)
    ap.add_argument("--windows", type=int, default=10, help="interleaved FP4/BF16 timing windows of 300 ms")
    ap.add_argument("--workload", default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bf16", action="store_true")
    ap.add_argument("--no-paper-shapes", action="store_true", help="skip the paper's reported shapes")
    ap.add_argument("--traffic-run", action="store_true",
                    help="for rocprofv3 --pmc passes: one 256 MiB device copy (counter calibration), "
                         "then one forward launch; prints no JSON")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the traffic file from the two --traffic-run counter CSVs (no GPU use)")
    args = ap.parse_args()
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the forward shards over (batch, head) with no communication "
              "and nothing here uses a second GPU; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads
    import paper_2609_04105_amd as fa

    name = args.workload or workloads.BENCH_WORKLOAD
    w = workloads.WORKLOADS[name]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    q_cpu, k_cpu, v_cpu = workloads.generate(w)
    q, k, v = (t.to(dev) for t in (q_cpu, k_cpu, v_cpu))
    torch.cuda.synchronize()

    ops = fa.quantize_qkv(q, k, v)
    out = torch.empty((w.B, w.H, w.N, w.d), dtype=torch.float32, device=dev)
    q16, k16 = q.to(torch.bfloat16), k.to(torch.bfloat16)
    vt16 = fa.transpose_bf16(v.to(torch.bfloat16))
    out16 = torch.empty_like(out)

    if args.traffic_run:
        src = torch.empty(64 << 20, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)                      # reads and writes exactly 256 MiB
        torch.cuda.synchronize()
        fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out)
        torch.cuda.synchronize()
        print(f"traffic run done: copy 268435456 B, one forward on {name}", flush=True)
        return

    def fp4_step():
        fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out)

    def bf16_step():
        fa.forward_bf16(q16, k16, vt16, softmax_scale=w.softmax_scale, out=out16)

    def quant_step():
        fa.quantize_qkv(q, k, v)

    # warmup (the BF16 kernel warms up in its first timing window)
    for _ in range(args.warmup):
        fp4_step()
    torch.cuda.synchronize()

    # the timed region: exactly `steps` forward steps, synchronized on both sides
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(args.steps):
        fp4_step()
    ev1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_start) * 1e3
    fp4_ms = ev0.elapsed_time(ev1) / args.steps

    # the paper's speedup convention: FP4 and BF16 windows interleaved
    pair = {"fp4": fp4_step}
    if not args.no_bf16:
        pair["bf16"] = bf16_step
    med, _ = _time_windows(torch, pair, 300.0, args.windows)
    fns = {}
    # native-exponential mixing (k of the 16 pairs of each 32-key block): the
    # `accurate` policy's quarter and the exp2-only route, same inputs
    for kx in EX2_SWEEP:
        fns[f"ex2_{kx}"] = (lambda kx=kx: fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out,
                                                           ex2_pairs=kx))
    # the sampled QK guard (Alg. 3) on anchor-ordered K and V, the paper's (M, L) = (110, 16)
    ops_anchored = fa.quantize_qkv(q, k, v, anchored=True)
    fns["guard"] = lambda: fa.forward_mxfp4(*ops_anchored, softmax_scale=w.softmax_scale, out=out,
                                            guard=GUARD_ML)
    # FP8 (E4M3) P and V: the paper's accuracy control and training route
    ops8 = fa.quantize_qkv(q, k, v, pv_fp8=True)
    fns["fp8pv"] = lambda: fa.forward_mxfp4(*ops8, softmax_scale=w.softmax_scale, out=out, pv_fp8=True)
    # the causal forward with the row normaliser saved for a backward pass
    lse = torch.empty((w.B, w.H, w.N), dtype=torch.float32, device=dev)
    fns["causal"] = lambda: fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out, causal=True, lse=lse)
    med.update(_time_windows(torch, fns, 150.0, 3)[0])
    qms, _ = _time_windows(torch, {"quant": quant_step}, 50.0, 3)

    flops = w.flops
    tflops = flops / (fp4_ms * 1e-3) / 1e12
    bf16_tflops = flops / (med["bf16"] * 1e-3) / 1e12 if "bf16" in med else None
    traffic = _traffic()
    clk = measured_clock_ghz(torch, fa, ops, w)
    peak_clk = MXFP4_PEAK_TFLOPS * clk / SPEC_CLOCK_GHZ
    stream_blocks = min(1024, ops[0].numel() // (256 * 64))  # 64 operand bytes per thread
    stream = sustained_mfma_tflops(torch, fa, ops[2].reshape(-1), ops[0].reshape(-1), blocks=stream_blocks) \
        if stream_blocks >= 1 else None
    roof = {
        "bound": "mfma",
        "achieved": round(tflops, 2),
        "peak": MXFP4_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(tflops / MXFP4_PEAK_TFLOPS, 4),
        "traffic": traffic,
        "kernel": "fwd_mxfp4_kernel<128, 8, false, 0, 0>",
        "measured_clock_ghz": round(clk, 3),
        "peak_at_measured_clock": round(peak_clk, 1),
        "frac_at_measured_clock": round(tflops / peak_clk, 4),
        "sustained_mfma_stream": round(stream, 1) if stream else None,
        "frac_of_sustained_mfma_stream": round(tflops / stream, 4) if stream else None,
        "algorithmic_flops_per_launch": flops,
    }
    line = {
        "metric": "MXFP4 attn fwd TFLOPS (4BHN^2d/t), % MXFP4 MFMA peak, speedup vs BF16",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(fp4_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "mxfp4",
        "data": "synthetic",
        "config": {"workload": name, "B": w.B, "H": w.H, "N": w.N, "d": w.d, "inputs": f"{w.dist} {w.dtype}",
                   "seed": w.seed, "softmax_scale": w.softmax_scale, "affine": [1.5, 1.2],
                   "output": "fp32", "parallelism": "single GPU"},
        "pct_mxfp4_peak": round(100 * tflops / MXFP4_PEAK_TFLOPS, 2),
        "bf16_tflops": None if bf16_tflops is None else round(bf16_tflops, 2),
        "bf16_pct_peak": None if bf16_tflops is None else round(100 * bf16_tflops / BF16_PEAK_TFLOPS, 2),
        "speedup_vs_bf16": None if "bf16" not in med else round(med["bf16"] / med["fp4"], 3),
        "fp4_ms_median_interleaved": round(med["fp4"], 5),
        "bf16_ms_median_interleaved": None if "bf16" not in med else round(med["bf16"], 5),
        "quantize_qkv_ms": round(qms["quant"], 5),
        "ex2_pairs_sweep": {str(kx): {"ms": round(med[f"ex2_{kx}"], 5),
                                      "tflops": round(flops / (med[f"ex2_{kx}"] * 1e-3) / 1e12, 2),
                                      "vs_affine": round(med["fp4"] / med[f"ex2_{kx}"], 3)} for kx in EX2_SWEEP},
        "guard_110_16": {"ms": round(med["guard"], 5), "tflops": round(flops / (med["guard"] * 1e-3) / 1e12, 2),
                         "vs_online": round(med["fp4"] / med["guard"], 3)},
        "fp8_pv": {"ms": round(med["fp8pv"], 5), "tflops": round(flops / (med["fp8pv"] * 1e-3) / 1e12, 2),
                   "vs_mxfp4_pv": round(med["fp4"] / med["fp8pv"], 3)},
        # visible (query, key) pairs only: 4 d B H N (N + 1) / 2 flop
        "causal_with_lse": {"ms": round(med["causal"], 5),
                            "tflops": round(2.0 * w.d * w.B * w.H * w.N * (w.N + 1) / (med["causal"] * 1e-3) / 1e12, 2),
                            "flops": "4 d B H N (N + 1) / 2"},
        "wall_ms_timed_region": round(wall_ms, 3),
        "roofline": roof,
        "gpu": torch.cuda.get_device_name(dev),
        "gfx_target": torch.cuda.get_device_properties(dev).gcnArchName,
        "kernel_source_sha256": _source_sha(),
    }
    if not args.no_paper_shapes and not args.no_bf16:
        line["paper_shapes"] = paper_shape_sweep(torch, fa)
    if not args.no_cpu_baseline:
        import numpy as np
        line["cpu_baseline"], o_ref = cpu_oracle_baseline(w, q_cpu, k_cpu, v_cpu)
        # parity of the timed launch on the rows the oracle computed (head (0, 0))
        fp4_step()
        torch.cuda.synchronize()
        got = out[0, 0, :len(o_ref)].double().cpu().numpy()
        rel = float(np.linalg.norm(got - o_ref) / np.linalg.norm(o_ref))
        cos = float(np.sum(got * o_ref) / (np.linalg.norm(got) * np.linalg.norm(o_ref)))
        line["parity"] = {"rows": int(len(o_ref)), "head": [0, 0], "o_rel_l2": rel, "o_cos": cos,
                          "gate": {"o_rel_l2_max": 2e-3, "o_cos_min": 0.9999},
                          "pass": bool(rel <= 2e-3 and cos >= 0.9999)}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
