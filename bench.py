"""Throughput of the Direct-P full-MXFP4 attention forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
    python bench.py --profile-run                  (one launch per route, for rocprofv3 passes)
    python bench.py --counter-summary P0 P1 P2 P3  (writes profiles/counters_routes.json)
    python bench.py --power-run                    (board power, clocks and the stream's occupancy sweep)

A step is one forward pass (QK on scaled FP4 matrix cores, Direct-P, PV, the
epilogue) over the whole workload with MXFP4 operands already resident in HBM;
the paper times the attention kernel on prequantized operands and excludes
quantization (its Sec. "Timed scope and operand contract").  The quantizer is
timed separately and reported in the same line.  The metric is the paper's
ops count 4 B H N^2 d per step (eq. hao-flops) over the step time.

Prints one JSON line.  Also reported: the same-design BF16 kernel on the same
inputs (windows interleaved with the FP4 ones, the paper's speedup
t_BF16 / t_FP4), the roofline of the forward kernel against the dense MXFP4
matrix peak (and, beside it, the shader clock the kernel holds when run back
to back, its rate and cycles per workgroup on the workload's codes and on
all-zero codes, and the rate a stream of FP4 matrix products alone sustains on
the workload's K and Q codes, two waves per SIMD), the quantizer's HBM
roofline, HBM traffic and hardware-counter figures per route from the committed
counter file (only while it matches the kernel sources), the other routes
(native-exponential pairs, the sampled guard, FP8 P/V, causal with LSE), the
other four workloads, both kernels on the shapes the paper reports (D128 and
D64) next to the paper's printed rates, and the CPU oracle timed on a seeded
sample of the workload's rows.  The defaults follow the paper's timing protocol (Sec.
"Operator benchmark suites"): 240 warmup steps (over 300 ms), 2200 timed steps
(about 3 s), and ten interleaved 300 ms windows of each of the FP4 and BF16
kernels.
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
COUNTER_FILE = os.path.join(ROOT, "profiles", "counters_routes.json")
CSRC = os.path.join(ROOT, "paper_2609_04105_amd", "csrc")
KERNEL_SOURCES = [os.path.join(CSRC, f) for f in ("fwd_mxfp4.hpp", "fwd_mxfp4.hip", "gfx950.hpp", "launch.hpp")]
BF16_SOURCES = [os.path.join(CSRC, f) for f in ("fwd_bf16.hip", "gfx950.hpp", "launch.hpp")]


def _source_sha(paths=None):
    """Hash of kernel sources with comments and blank lines removed, so that the
    committed counters stay attached to the code they measured (default: the
    MXFP4 forward's sources)."""
    h = hashlib.sha256()
    for path in (paths or KERNEL_SOURCES):
        with open(path) as f:
            for line in f:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()


# Routes whose counters are committed (one launch each, in this order, under
# ``--profile-run``): (label, inputs, kernel family, route options).  Inputs are a
# workload name or a paper shape "d64_b1h64_n32768" (N(0, 1) bf16 drawn on the GPU).
PROFILE_ROUTES = [
    ("online", "long_b1h32_n16384_d128", "fp4", {}),
    ("ex2_1", "long_b1h32_n16384_d128", "fp4", {"ex2_pairs": 1}),
    ("ex2_2", "long_b1h32_n16384_d128", "fp4", {"ex2_pairs": 2}),
    ("ex2_4", "long_b1h32_n16384_d128", "fp4", {"ex2_pairs": 4}),
    ("ex2_16", "long_b1h32_n16384_d128", "fp4", {"ex2_pairs": 16}),
    ("guard_110_16", "long_b1h32_n16384_d128", "fp4", {"guard": (110, 16)}),
    ("causal_lse", "long_b1h32_n16384_d128", "fp4", {"causal": True, "lse": True}),
    ("fp8_pv", "long_b1h32_n16384_d128", "fp4", {"pv_fp8": True}),
    ("bf16", "long_b1h32_n16384_d128", "bf16", {}),
    ("online", "outlier_b2h16_n4096_d128", "fp4", {}),
    ("online", "student_t_b1h32_n8192_d128", "fp4", {}),
    ("online", "d64_b1h64_n32768", "fp4", {}),
    ("bf16", "d64_b1h64_n32768", "bf16", {}),
]
PASSES = [
    "SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_VALU_TRANS_F32 SQ_INSTS_VALU_CVT SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_LDS "
    "SQ_BUSY_CYCLES SQ_WAVE_CYCLES GRBM_GUI_ACTIVE",
    "SQ_INSTS_VALU_FMA_F32 SQ_ACTIVE_INST_VALU SQ_WAIT_INST_ANY SQ_VALU_MFMA_COEXEC_CYCLES SQ_INSTS_SALU "
    "SQ_LDS_BANK_CONFLICT SQ_ACTIVE_INST_LDS SQ_WAIT_INST_LDS GRBM_GUI_ACTIVE",
    "FETCH_SIZE",
    "WRITE_SIZE",
]
N_SIMD = 1024   # 256 CUs x 4 SIMDs
N_XCD = 8


def _shape_of(inputs):
    """(B, H, N, d, seed-or-None) of a route's inputs."""
    import workloads
    if inputs in workloads.WORKLOADS:
        w = workloads.WORKLOADS[inputs]
        return w.B, w.H, w.N, w.d, w
    import re
    m = re.fullmatch(r"d(\d+)_b(\d+)h(\d+)_n(\d+)", inputs)
    if m is None:
        raise ValueError(f"unknown route inputs {inputs!r}")
    d, b, h, n = (int(x) for x in m.groups())
    return b, h, n, d, None


def _route_inputs(torch, fa, inputs, cache):
    """bf16/fp32 q, k, v on the GPU and their MXFP4 operands (cached per inputs)."""
    if inputs not in cache:
        import workloads
        B, H, N, d, w = _shape_of(inputs)
        if w is not None:
            q, k, v = (t.cuda() for t in workloads.generate(w))
        else:
            g = torch.Generator(device="cuda").manual_seed(21)
            q, k, v = (torch.randn((B, H, N, d), device="cuda", generator=g).to(torch.bfloat16) for _ in range(3))
        cache[inputs] = (q, k, v, {})
    return cache[inputs]


def _route_call(torch, fa, label, inputs, family, opts, cache):
    """A no-argument callable that launches one route's forward (operands prepared)."""
    q, k, v, ops_cache = _route_inputs(torch, fa, inputs, cache)
    B, H, N, d, _ = _shape_of(inputs)
    scale = 1.0 / math.sqrt(d)
    out = torch.empty((B, H, N, d), dtype=torch.float32, device="cuda")
    if family == "bf16":
        return lambda: fa.forward_bf16(q, k, v, softmax_scale=scale, out=out)
    key = "anchored" if "guard" in opts else ("fp8" if opts.get("pv_fp8") else "plain")
    if key not in ops_cache:
        ops_cache[key] = fa.quantize_qkv(q, k, v, anchored=key == "anchored", pv_fp8=key == "fp8")
    ops = ops_cache[key]
    kw = dict(opts)
    if kw.pop("lse", False):
        kw["lse"] = torch.empty((B, H, N), dtype=torch.float32, device="cuda")
    return lambda: fa.forward_mxfp4(*ops, softmax_scale=scale, out=out, **kw)


def profile_run(torch, fa):
    """For rocprofv3 passes: a 256 MiB device copy (the traffic counters'
    calibration), then one launch of every route of PROFILE_ROUTES, in order."""
    src = torch.empty(64 << 20, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    cache = {}
    calls = [_route_call(torch, fa, *r, cache) for r in PROFILE_ROUTES]
    torch.cuda.synchronize()
    for (label, inputs, family, _), fn in zip(PROFILE_ROUTES, calls):
        fn()
        torch.cuda.synchronize()
        print(f"profile run: {label} on {inputs} ({family}) launched", flush=True)


def _route_scores(inputs, opts):
    """(scores, flop) of one launch: B H N^2 score entries (causal: the visible
    pairs B H N (N + 1) / 2) and 4 d per score."""
    B, H, N, d, _ = _shape_of(inputs)
    scores = B * H * N * (N + 1) / 2 if opts.get("causal") else B * H * N * N
    return scores, 4.0 * d * scores


def counter_summary(out_path, csv_paths, routes=None):
    """Write the per-route counter file from the CSVs of the ``--profile-run``
    passes (PASSES, in order).  Forward-kernel dispatches are matched to
    PROFILE_ROUTES by dispatch order; the traffic counters are scaled by what they
    read for the 256 MiB device copy of the same run."""
    import csv
    routes = PROFILE_ROUTES if routes is None else routes
    per_pass = []
    for path in csv_paths:
        disp = {}
        with open(path) as f:
            for r in csv.DictReader(f):
                d = disp.setdefault(int(r["Dispatch_Id"]), {"kernel": r["Kernel_Name"], "c": {},
                                                              "vgpr": int(r["VGPR_Count"]),
                                                              "agpr": int(r["Accum_VGPR_Count"]),
                                                              "lds": int(r["LDS_Block_Size"]),
                                                              "scratch": int(r["Scratch_Size"])})
                d["c"][r["Counter_Name"]] = d["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        order = sorted(disp)
        fwd = [disp[i] for i in order if "fwd_mxfp4_kernel" in disp[i]["kernel"] or "fwd_bf16_kernel" in disp[i]["kernel"]]
        copy = [disp[i] for i in order if "copyBuffer" in disp[i]["kernel"]]
        if len(fwd) != len(routes) or len(copy) != 1:
            raise SystemExit(f"{path}: {len(fwd)} forward dispatches (expected {len(routes)}), "
                             f"{len(copy)} copies (expected 1)")
        per_pass.append((fwd, copy[0]))
    copy_kib = (256 << 20) / 1024
    records = []
    for i, (label, inputs, family, opts) in enumerate(routes):
        c = {}
        for fwd, copy in per_pass:
            c.update(fwd[i]["c"])
        k = per_pass[0][0][i]
        scores, flop = _route_scores(inputs, opts)
        B, H, N, d, _ = _shape_of(inputs)
        rec = {"label": label, "inputs": inputs, "family": family, "options": {kk: list(vv) if isinstance(vv, tuple)
                                                                               else vv for kk, vv in opts.items()},
               "kernel": k["kernel"].replace("(anonymous namespace)::", "").split("(")[0].replace("void ", ""),
               "vgpr": k["vgpr"], "agpr": k["agpr"], "lds_bytes": k["lds"], "scratch_bytes": k["scratch"],
               "counters": c, "scores": scores, "flop": flop}
        der = {}
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c and "GRBM_GUI_ACTIVE" in c:
            der["mfma_busy_pct"] = 100.0 * c["SQ_VALU_MFMA_BUSY_CYCLES"] / (c["GRBM_GUI_ACTIVE"] / N_XCD * N_SIMD)
        if "SQ_INSTS_VALU" in c and "SQ_INSTS_MFMA" in c:
            der["valu_non_mfma_per_score"] = (c["SQ_INSTS_VALU"] - c["SQ_INSTS_MFMA"]) * 64 / scores
            der["mfma_per_score"] = c["SQ_INSTS_MFMA"] * 64 / scores
        for name, key in (("SQ_INSTS_VALU_TRANS_F32", "trans_per_score"), ("SQ_INSTS_VALU_CVT", "cvt_per_score"),
                          ("SQ_INSTS_VALU_FMA_F32", "fma_f32_per_score"), ("SQ_INSTS_LDS", "lds_insts_per_score"),
                          ("SQ_INSTS_SALU", "salu_per_score")):
            if name in c:
                der[key] = c[name] * 64 / scores
        if "SQ_WAIT_INST_ANY" in c and "SQ_WAVE_CYCLES" in c:
            der["wait_inst_any_pct_of_wave_cycles"] = 100.0 * c["SQ_WAIT_INST_ANY"] / c["SQ_WAVE_CYCLES"]
        if "SQ_LDS_BANK_CONFLICT" in c and "SQ_ACTIVE_INST_LDS" in c and c["SQ_ACTIVE_INST_LDS"]:
            der["lds_bank_conflict_pct_of_lds_active"] = 100.0 * c["SQ_LDS_BANK_CONFLICT"] / c["SQ_ACTIVE_INST_LDS"]
        if "FETCH_SIZE" in c and "WRITE_SIZE" in c:
            fetch_copy = [cp["c"]["FETCH_SIZE"] for _, cp in per_pass if "FETCH_SIZE" in cp["c"]][0]
            write_copy = [cp["c"]["WRITE_SIZE"] for _, cp in per_pass if "WRITE_SIZE" in cp["c"]][0]
            der["fetch_bytes"] = c["FETCH_SIZE"] * 1024 * (copy_kib / fetch_copy)
            der["write_bytes"] = c["WRITE_SIZE"] * 1024 * (copy_kib / write_copy)
            der["hbm_bytes"] = der["fetch_bytes"] + der["write_bytes"]
            der["copy_scale"] = {"fetch": copy_kib / fetch_copy, "write": copy_kib / write_copy}
        if family == "fp4":
            mx = 1 if opts.get("pv_fp8") else 0.5
            der["algorithmic_bytes"] = B * H * (N * d * (2 * (0.5 + 1 / 32) + mx + 1 / 32) + 4 * N * d) + (
                4 * B * H * N if opts.get("lse") else 0)
        else:
            der["algorithmic_bytes"] = B * H * (3 * 2 * N * d + 4 * N * d)
        rec["derived"] = der
        rec["source_sha256"] = _source_sha(KERNEL_SOURCES if family == "fp4" else BF16_SOURCES)
        records.append(rec)
    res = {"routes": records, "passes": PASSES,
           "commands": [f"timeout -s KILL 120 rocprofv3 --pmc {p} --output-format csv -d <dir{i}> -o p{i} -- "
                        f"python bench.py --profile-run" for i, p in enumerate(PASSES)] +
                       ["python bench.py --counter-summary " + " ".join(f"<dir{i}>/p{i}_counter_collection.csv"
                                                                         for i in range(len(PASSES)))]}
    with open(out_path, "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps({"routes": [(r["label"], r["inputs"], r["derived"]) for r in records]}, indent=1))
    return res


def _route_counters(label, inputs):
    """Derived counter figures of a route from the committed counter file, if they
    were taken on the current source of that route's kernel; else None."""
    try:
        with open(COUNTER_FILE) as f:
            res = json.load(f)
    except (OSError, ValueError):
        return None
    for r in res.get("routes", []):
        if r["label"] == label and r["inputs"] == inputs:
            sha = _source_sha(KERNEL_SOURCES if r["family"] == "fp4" else BF16_SOURCES)
            return dict(r["derived"], kernel=r["kernel"]) if r.get("source_sha256") == sha else None
    return None


def quantizer_roofline(torch, fa, qkv, qkv_ms):
    """HBM roofline of the input quantizer (outside the timed forward, as in the
    paper).  Algorithmic bytes per element: the bf16 input read once (2) and the
    E2M1 code (1/2) plus 1/32 of an E8M0 byte written.  Each kernel is timed on Q,
    K and V in turn (three tensors, more than the 256 MB Infinity Cache when each
    is as large as the long workload's), so every call reads its input from HBM:
    the rows kernel (blocks along d: Q and K) and the V^T kernel (blocks along the
    sequence, transposed output)."""
    n = qkv[0].numel()
    per_elem = 2 + 0.5 + 1 / 32
    if qkv[0].dtype != torch.bfloat16:
        return None
    turn = {"rows": 0, "vt": 0}

    def call(axis, key):
        x = qkv[turn[key] % 3]
        turn[key] += 1
        fa.quantize_mxfp4(x, axis=axis)

    med, _ = _time_windows(torch, {"rows": lambda: call(-1, "rows"), "vt": lambda: call(-2, "vt")}, 50.0, 5)

    def entry(us, nbytes):
        gbs = nbytes / (us * 1e-6) / 1e9
        return {"us": round(us, 2), "algorithmic_bytes": int(nbytes), "achieved": round(gbs, 1),
                "frac": round(gbs / HBM_PEAK_GBS, 4)}

    return {"bound": "hbm", "peak": HBM_PEAK_GBS, "unit": "GB/s", "bytes_per_element": per_elem,
            "rows_kernel": entry(med["rows"] * 1e3, n * per_elem),
            "vt_kernel": entry(med["vt"] * 1e3, n * per_elem),
            "quantize_qkv": entry(qkv_ms * 1e3, 3 * n * per_elem)}


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


def _sustained_clock(torch, fa, ops, w, out, seconds):
    """Run the timed forward back to back for ``seconds`` on the operands ``ops``;
    over the second half, launches with the workgroup clock record give the
    kernel's shader clock and the median shader cycles per workgroup.  Returns
    (TFLOP/s over every launch of the window, clock in GHz, cycles per workgroup)."""
    no_rows = torch.zeros(0, dtype=torch.int64, device=ops[0].device)
    fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    t0, n, recs = time.time(), 0, []
    while time.time() - t0 < seconds:
        for _ in range(8):
            fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out)
        n += 8
        if time.time() - t0 > seconds / 2:
            # the record stays on the device until the window ends
            recs.append(fa.debug_directp_mxfp4(*ops, no_rows, softmax_scale=w.softmax_scale,
                                               wg_clock=True)["wg_clock"])
            n += 1
        torch.cuda.synchronize()
    if not recs:   # a window too short for a record in its second half
        recs.append(fa.debug_directp_mxfp4(*ops, no_rows, softmax_scale=w.softmax_scale, wg_clock=True)["wg_clock"])
        n += 1
    e.record()
    torch.cuda.synchronize()
    c = torch.cat([r.cpu() for r in recs]).double()
    c = c[c[:, 0] > 0]   # rows past the launch's workgroup count stay zero
    return (w.flops * n / (s.elapsed_time(e) * 1e-3) / 1e12, float(c[:, 0].sum() / (c[:, 1].sum() / 100e6) / 1e9),
            float(c[:, 0].median()))


def clock_vs_data(torch, fa, ops, w, out, seconds=1.5):
    """The timed kernel on the workload's codes and on all-zero Q, K and V^T codes
    (the same scales, instructions, copies and LDS reads; the products see no data
    activity), one sustained window each: how much of the gap to the spec peak is
    the schedule (cycles per workgroup) and how much the clock the chip holds on
    the data."""
    zero = list(ops)
    for i in (0, 2, 4):
        zero[i] = torch.zeros_like(ops[i])
    res = {}
    for label, o in (("workload_codes", ops), ("zero_codes", tuple(zero))):
        tf, clk, cyc = _sustained_clock(torch, fa, o, w, out, seconds)
        res[label] = {"tflops": round(tf, 1), "frac_of_peak": round(tf / MXFP4_PEAK_TFLOPS, 4),
                      "kernel_clock_ghz": round(clk, 3), "cycles_per_workgroup": round(cyc)}
    for r in res.values():
        # the rate against the spec peak scaled to the clock the kernel ran at
        r["frac_at_kernel_clock"] = round(r["tflops"] / (MXFP4_PEAK_TFLOPS * r["kernel_clock_ghz"] / SPEC_CLOCK_GHZ), 4)
    res["seconds_each"] = seconds
    return res


def stream_blocks(torch):
    """Workgroups of the matrix-product stream: two per CU (four-wave workgroups,
    so two waves per SIMD, all resident in one round).  The stream's rate falls
    with three or more waves per SIMD (on zero bytes 9.7 PFLOP/s at two, 7.0 at
    three, 6.3 when four are asked for and three fit), so this is the launch
    that shows the matrix unit's ceiling."""
    return 2 * torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count


def sustained_mfma_tflops(torch, fa, a_codes, b_codes, blocks=512, iters=200000, launches=7):
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
        bf = (q, k, v)
        out = torch.empty((1, H, S, d), dtype=torch.float32, device="cuda")
        scale = 1.0 / math.sqrt(d)
        fns = {"fp4": lambda: fa.forward_mxfp4(*ops, softmax_scale=scale, out=out),
               "bf16": lambda: fa.forward_bf16(*bf, softmax_scale=scale, out=out)}
        for fn in fns.values():
            fn()
        med = _time_windows(torch, fns, 100.0, 3)[0]
        flop = 4.0 * H * S * S * d
        res.append({"shape": f"B1/S{S}/H{H}/D{d}", "tflops": round(flop / (med["fp4"] * 1e-3) / 1e12, 1),
                    "bf16_tflops": round(flop / (med["bf16"] * 1e-3) / 1e12, 1),
                    "speedup_vs_bf16": round(med["bf16"] / med["fp4"], 3),
                    "paper_nvmx_tflops": {"gb200": gb200, "b300": b300}})
        del q, k, v, ops, bf, out
    return res


def cpu_oracle_baseline(w, q, k, v, target_s=15.0):
    """Time the oracle (as it stands) on a bounded, seeded sample of the workload's
    query rows (CPU tensors q, k, v [B, H, N, d]): per (batch, head) its own MXFP4
    quantization of K, V and the sampled Q rows, then the Direct-P forward of those
    rows.  Heads run on a pool of host threads, each with a single-threaded BLAS.
    First the 4096 rows the parity tests check; then further passes over the next rows
    of the same seeded permutation, each sized from the previous one, until the
    passes together take about ``target_s`` seconds (each pass quantizes its heads'
    K and V again; at most 64 times the first pass's rows).  Returns the record and
    (rows, O) for the parity check of the timed launch."""
    import numpy as np
    import workloads
    from concurrent.futures import ThreadPoolExecutor
    from oracle import directp, mxfp4
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        info = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')}"
    except Exception:  # threadpoolctl missing: BLAS threads as configured
        threadpool_limits = None
    workers = max(1, min(16, len(os.sched_getaffinity(0))))

    def run(rows):
        heads = rows // w.N

        def one_head(bh):
            b, h = divmod(int(bh), w.H)
            sel = np.nonzero(heads == bh)[0]
            q64, k64, v64 = (workloads.as_f64(t[b:b + 1, h:h + 1])[0, 0] for t in (q, k, v))
            qc, qs = mxfp4.quantize(q64[rows[sel] % w.N], axis=-1)
            kc, ks = mxfp4.quantize(k64, axis=-1)
            vc, vs = mxfp4.quantize(v64, axis=-2)
            return sel, directp.forward_rows(qc, qs, kc, ks, vc, vs, np.arange(len(sel)), w.softmax_scale,
                                             want_codes=False)["O"]

        out = np.zeros((len(rows), w.d))
        t0 = time.perf_counter()
        limit = threadpool_limits(1, user_api="blas") if threadpool_limits else None
        try:
            with ThreadPoolExecutor(max_workers=workers) as ex:
                for sel, o in ex.map(one_head, np.unique(heads)):
                    out[sel] = o
        finally:
            if limit is not None:
                limit.unregister() if hasattr(limit, "unregister") else None
        return out, time.perf_counter() - t0

    first = workloads.sampled_rows(w)
    out, dt = run(first)
    rows, last_n, last_dt = first, len(first), dt
    # Each further pass is sized from the previous pass's time per row, which
    # includes that pass's quantization and so overstates the cost of a row.
    while dt < 0.7 * target_s and len(rows) < w.rows and len(rows) < 64 * len(first):
        extra = int(last_n * (target_s - dt) / last_dt) // 4096 * 4096
        extra = min(max(extra, 4096), w.rows - len(rows), 64 * len(first) - len(rows))
        more = np.setdiff1d(workloads.sampled_rows(w, len(rows) + extra), rows)
        o, t = run(more)
        rows, out, dt = np.concatenate([rows, more]), np.concatenate([out, o]), dt + t
        last_n, last_dt = len(more), t
    flops = 4.0 * len(rows) * w.N * w.d
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": workers,
        "kind": "oracle",
        "sample": f"{len(rows)} seeded sampled query rows of {w.name} over its {len(np.unique(rows // w.N))} heads "
                  f"(all {w.N} keys): the {len(first)} rows of the parity tests, then the next {len(rows) - len(first)}"
                  f" of the same seeded permutation in further passes; each pass includes the oracle's own MXFP4 "
                  f"quantization of each head's K, V and sampled Q rows; {workers} host threads (one per head at a "
                  f"time, single-threaded BLAS); {dt:.1f} s",
        "blas": blas,
        "seconds": round(dt, 2),
        "full_workload_estimate_s": round(dt * w.rows / len(rows), 1),
    }, (rows, out)


def graph_us_per_launch(torch, fns, launches=50, replays=20):
    """Microseconds per launch of each fn with the host's launch cost taken out:
    ``launches`` back-to-back calls captured once in a HIP graph (torch.cuda.graph)
    and replayed; median over ``replays`` timed replays."""
    res = {}
    for name, fn in fns.items():
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(launches):
                fn()
        graph.replay()
        torch.cuda.synchronize()
        times = []
        for _ in range(replays):
            start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            start.record()
            graph.replay()
            end.record()
            torch.cuda.synchronize()
            times.append(start.elapsed_time(end) * 1e3 / launches)
        res[name] = sorted(times)[len(times) // 2]
        del graph
    return res


def other_configs(torch, fa, exclude):
    """The remaining workloads: the forward and the BF16 kernel timed in
    interleaved windows on each one's own inputs.  The two small ones are
    launch-bound (microseconds of launch and fill against sub-microsecond
    matrix work at peak); the two large ones are matrix-bound points with the
    roofline fraction and, where committed counters match the kernel source,
    their HBM traffic.  For the launch-bound ones the per-launch time of a
    captured HIP graph of back-to-back launches is reported beside the
    per-call time."""
    import workloads
    res = []
    for name, w in workloads.WORKLOADS.items():
        if name == exclude:
            continue
        q, k, v = (t.cuda() for t in workloads.generate(w))
        ops = fa.quantize_qkv(q, k, v)
        out = torch.empty((w.B, w.H, w.N, w.d), dtype=torch.float32, device="cuda")
        bf = (q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16))
        fns = {"fp4": lambda: fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out),
               "bf16": lambda: fa.forward_bf16(*bf, softmax_scale=w.softmax_scale, out=out)}
        for fn in fns.values():
            fn()
        med = _time_windows(torch, fns, 100.0, 5)[0]
        tflops = w.flops / (med["fp4"] * 1e-3) / 1e12
        rec = {"workload": name, "B": w.B, "H": w.H, "N": w.N, "d": w.d, "inputs": f"{w.dist} {w.dtype}",
               "seed": w.seed, "ms": round(med["fp4"], 5), "tflops": round(tflops, 2),
               "frac": round(tflops / MXFP4_PEAK_TFLOPS, 4),
               "bf16_tflops": round(w.flops / (med["bf16"] * 1e-3) / 1e12, 2),
               "speedup_vs_bf16": round(med["bf16"] / med["fp4"], 3),
               "us_at_mxfp4_peak": round(w.flops / (MXFP4_PEAK_TFLOPS * 1e12) * 1e6, 4)}
        if w.flops < 1e10:
            rec["bound"] = "launch"
            rec["us_per_launch"] = round(med["fp4"] * 1e3, 3)
            g_us = graph_us_per_launch(torch, fns)
            rec["graph_us_per_launch"] = {k: round(v, 3) for k, v in g_us.items()}
            rec["graph_tflops"] = round(w.flops / (g_us["fp4"] * 1e-6) / 1e12, 2)
            rec["graph_speedup_vs_bf16"] = round(g_us["bf16"] / g_us["fp4"], 3)
        else:
            rec["bound"] = "mfma"
            c = _route_counters("online", name)
            if c is not None:
                rec["traffic"] = round(c["hbm_bytes"])
                rec["algorithmic_bytes"] = c["algorithmic_bytes"]
                rec["hbm_gbs"] = round(c["hbm_bytes"] / (med["fp4"] * 1e-3) / 1e9, 1)
                rec["mfma_busy_pct_counters"] = round(c["mfma_busy_pct"], 2)
            else:
                rec["traffic"] = None
        res.append(rec)
        del q, k, v, ops, out, bf
    return res


def _counter_view(c, ms):
    """The figures of a route's counter record that the bench line carries."""
    if c is None:
        return None
    keys = ("mfma_busy_pct", "valu_non_mfma_per_score", "trans_per_score", "cvt_per_score", "fma_f32_per_score",
            "lds_insts_per_score", "wait_inst_any_pct_of_wave_cycles", "hbm_bytes", "algorithmic_bytes")
    v = {key: (round(c[key], 4) if isinstance(c[key], float) else c[key]) for key in keys if key in c}
    if "hbm_bytes" in c:
        v["hbm_gbs"] = round(c["hbm_bytes"] / (ms * 1e-3) / 1e9, 1)
    return v


_SMI_SAMPLER = r"""
import json, os, subprocess, sys, time
parent = os.getppid()
with open(sys.argv[1], "a") as f:
    while os.getppid() == parent:   # ends with the process that started it
        t = time.time()
        try:
            r = subprocess.run(["amd-smi", "metric", "--power", "--clock", "--temperature", "--json"],
                               capture_output=True, text=True, timeout=30)
            out = r.stdout
        except Exception as e:
            out = json.dumps({"error": str(e)[:200]})
        f.write(json.dumps({"t": t, "out": out}) + "\n")
        f.flush()
        time.sleep(0.2)
"""


def start_power_sampler(path):
    """Start the amd-smi sampler as a child process (before this process makes
    any HIP call): every ~0.2 s it appends a timestamped reading of every card
    to ``path``.  amd-smi is only read: power, clocks, temperature."""
    import subprocess
    return subprocess.Popen([sys.executable, "-c", _SMI_SAMPLER, path], stdout=subprocess.DEVNULL,
                            stderr=subprocess.DEVNULL)


def _smi_cards(text):
    """Per card of one amd-smi JSON reading: socket power (W), the shader clock of
    each XCD (MHz) and the hotspot temperature (C); None where not reported."""
    data = json.loads(text)
    cards = data["gpu_data"] if isinstance(data, dict) else data
    res = []
    for g in cards:
        def val(x):
            return x.get("value") if isinstance(x, dict) else None
        clocks = [val(c.get("clk", {})) for key, c in g.get("clock", {}).items() if key.startswith("gfx_")]
        res.append({"gpu": g.get("gpu"), "power_w": val(g.get("power", {}).get("socket_power")),
                    "gfx_mhz": [c for c in clocks if c is not None],
                    "hotspot_c": val(g.get("temperature", {}).get("hotspot"))})
    return res


def _stop_sampler(sampler):
    if sampler.poll() is None:
        sampler.terminate()
        sampler.wait(timeout=30)


def board_readings(path, t0, t1):
    """Medians of the amd-smi readings taken inside [t0, t1] (wall clock) of the
    card whose power is highest there: socket power, XCD shader clocks, hotspot
    temperature.  None if the window holds no reading."""
    cards_by_time = []
    try:
        with open(path) as f:
            for line in f:
                try:
                    rec = json.loads(line)
                    if t0 <= rec["t"] <= t1:
                        cards_by_time.append(_smi_cards(rec["out"]))
                except (ValueError, KeyError, TypeError):
                    continue   # a line still being written, or a failed reading
    except OSError:
        return None
    if not cards_by_time:
        return None

    def med(xs):
        xs = sorted(x for x in xs if x is not None)
        return xs[len(xs) // 2] if xs else None
    n = max(len(c) for c in cards_by_time)
    card = max(range(n), key=lambda i: med([c[i]["power_w"] for c in cards_by_time if len(c) > i]) or 0)
    rows = [c[card] for c in cards_by_time if len(c) > card]
    clocks = [x for r in rows for x in r["gfx_mhz"]]
    return {"samples": len(rows), "socket_power_w_median": med([r["power_w"] for r in rows]),
            "gfx_clock_mhz_median": med(clocks), "hotspot_c_max": max((r["hotspot_c"] for r in rows
                                                                      if r["hotspot_c"] is not None), default=None),
            "source": "amd-smi metric (read-only), sampled during the timed region"}


def power_run(torch, fa, sampler, sample_path, seconds=4.0):
    """Board power, shader clocks and hotspot temperature (amd-smi readings taken
    by ``sampler``) while each load runs back to back for about ``seconds``: the
    card idle; the FP4 matrix-product stream (four independent 32x32x64 products
    per thread, nothing else) on zero bytes, on a constant byte (every code 1.0),
    on random bytes and on the long workload's K and Q codes; the MXFP4 forward on the long workload's
    codes and on all-zero codes (the same instructions, copies and LDS reads); the BF16 kernel on the
    long workload.  Then the stream's rate at one to four workgroups per CU.
    Prints one JSON line: per load the delivered TFLOP/s and the medians of the
    readings, taken while it ran, of the card whose power rose the most under the
    forward, and the stream's rate per occupancy."""
    import workloads
    w = workloads.WORKLOADS[workloads.BENCH_WORKLOAD]
    q, k, v = (t.cuda() for t in workloads.generate(w))
    ops = fa.quantize_qkv(q, k, v)
    bf = tuple(t.to(torch.bfloat16) for t in (q, k, v))
    out = torch.empty((w.B, w.H, w.N, w.d), dtype=torch.float32, device="cuda")
    blocks, iters = stream_blocks(torch), 200000
    nbytes = blocks * 256 * 64
    stream_flop = blocks * 4 * iters * 4 * 2.0 * 32 * 32 * 64
    g = torch.Generator(device="cuda").manual_seed(5)
    operands = {
        "zero": (torch.zeros((nbytes,), dtype=torch.uint8, device="cuda"),) * 2,
        "constant": (torch.full((nbytes,), 0x22, dtype=torch.uint8, device="cuda"),) * 2,
        "random": tuple(torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda", generator=g)
                        for _ in range(2)),
        "workload": (ops[2].reshape(-1)[:nbytes], ops[0].reshape(-1)[:nbytes]),
    }
    loads = [("idle", None, 0.0)]
    for kind, (a, b) in operands.items():
        loads.append((f"mfma_stream_{kind}", lambda a=a, b=b: fa.debug_mfma_stream(a, b, blocks, iters), stream_flop))
    loads.append(("mxfp4_forward", lambda: fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out), w.flops))
    zero_ops = list(ops)
    for i in (0, 2, 4):
        zero_ops[i] = torch.zeros_like(ops[i])
    loads.append(("mxfp4_forward_zero_codes",
                  lambda: fa.forward_mxfp4(*zero_ops, softmax_scale=w.softmax_scale, out=out), w.flops))
    loads.append(("bf16_forward", lambda: fa.forward_bf16(*bf, softmax_scale=w.softmax_scale, out=out), w.flops))

    results = []
    for name, fn, flop in loads:
        if fn is not None:
            fn()
        torch.cuda.synchronize()
        calls = 0
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        t0 = time.time()
        while time.time() - t0 < seconds:
            if fn is None:
                time.sleep(0.05)
                continue
            fn()
            calls += 1
            if calls % 8 == 0:
                torch.cuda.synchronize()
        end.record()
        torch.cuda.synchronize()
        t1 = time.time()
        ms = start.elapsed_time(end)
        results.append({"load": name, "calls": calls, "window": (t0, t1),
                        "tflops": round(flop * calls / (ms * 1e-3) / 1e12, 1) if calls else None})
        _progress(f"power run: {name} done")
    _, clk, _ = _sustained_clock(torch, fa, ops, w, out, 1.5)
    # the stream's rate against its occupancy: one to three waves per SIMD, and
    # four asked for where three fit (a second, lone round), ~1.5 s each
    occupancy = []
    cus = torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count
    for kind in ("zero", "random"):
        a, b = operands[kind]
        for per_cu, label in ((1, "1 wave per SIMD"), (2, "2 waves per SIMD"), (3, "3 waves per SIMD"),
                              (4, "4 asked, 3 fit")):
            nb = per_cu * cus
            big = torch.cat([a] * per_cu) if per_cu > 1 else a
            it = iters * 2 // per_cu
            fa.debug_mfma_stream(big, big, nb, 1000)
            torch.cuda.synchronize()
            calls, flop_total = 0, 0.0
            start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            start.record()
            t0 = time.time()
            while time.time() - t0 < 1.5:
                _, f = fa.debug_mfma_stream(big, big, nb, it)
                calls += 1
                flop_total += f
                if calls % 4 == 0:
                    torch.cuda.synchronize()
            end.record()
            torch.cuda.synchronize()
            occupancy.append({"operands": kind, "workgroups": nb, "occupancy": label,
                              "tflops": round(flop_total / (start.elapsed_time(end) * 1e-3) / 1e12, 1)})
            del big
    _progress("power run: stream occupancy sweep done")
    time.sleep(0.5)
    sampler.terminate()
    sampler.wait(timeout=30)
    readings = []
    with open(sample_path) as f:
        for line in f:
            rec = json.loads(line)
            try:
                readings.append((rec["t"], _smi_cards(rec["out"])))
            except (ValueError, KeyError, TypeError):
                pass

    def med(xs):
        xs = sorted(x for x in xs if x is not None)
        return xs[len(xs) // 2] if xs else None

    def during(r, i, key):
        # readings started well inside the load's window (the tool takes a while)
        t0, t1 = r["window"]
        return [cards[i].get(key) for t, cards in readings if t0 + 0.5 <= t <= t1 - 0.5 and len(cards) > i]

    n_cards = max((len(c) for _, c in readings), default=0)
    fwd = next(r for r in results if r["load"] == "mxfp4_forward")
    idle = results[0]
    rise = [(med(during(fwd, i, "power_w")) or 0) - (med(during(idle, i, "power_w")) or 0) for i in range(n_cards)]
    card = max(range(n_cards), key=lambda i: rise[i]) if n_cards else None
    for r in results:
        if card is not None:
            pw = during(r, card, "power_w")
            clocks = [c for cs in during(r, card, "gfx_mhz") if cs for c in cs]
            hs = [x for x in during(r, card, "hotspot_c") if x is not None]
            r.update({"samples": len(pw), "socket_power_w_median": med(pw),
                      "socket_power_w_max": max((x for x in pw if x is not None), default=None),
                      "gfx_clock_mhz_median": med(clocks),
                      "gfx_clock_mhz_range": [min(clocks), max(clocks)] if clocks else None,
                      "hotspot_c_max": max(hs) if hs else None})
        del r["window"]
    print(json.dumps({"power_run": results, "stream_occupancy": occupancy, "card_index_in_tool": card,
                      "n_cards_listed": n_cards,
                      "forward_in_kernel_clock_ghz": round(clk, 3), "workload": w.name,
                      "load_seconds": seconds}), flush=True)


def _progress(msg):
    """One line on stderr per finished stage, so a long run shows where it is."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


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
    ap.add_argument("--no-other-configs", action="store_true", help="skip the other four workloads")
    ap.add_argument("--profile-run", action="store_true",
                    help="for rocprofv3 passes: one 256 MiB device copy (traffic calibration), then one launch "
                         "of every profiled route; prints no JSON")
    ap.add_argument("--no-clock-vs-data", action="store_true",
                    help="skip the sustained windows of the timed kernel on the workload's and on zero codes (a "
                         "traced run keeps the timed kernel's dispatches to the workload's codes)")
    ap.add_argument("--no-board", action="store_true",
                    help="do not sample board power and clocks (amd-smi) during the timed region")
    ap.add_argument("--power-run", action="store_true",
                    help="board power, clocks and hotspot temperature (amd-smi) while the matrix-product stream, "
                         "the MXFP4 forward and the BF16 kernel each run back to back; one JSON line")
    ap.add_argument("--counter-summary", nargs="+", metavar="CSV",
                    help="write the per-route counter file from the --profile-run counter CSVs, one per pass "
                         "in the order of PASSES (no GPU use)")
    args = ap.parse_args()
    if args.counter_summary:
        counter_summary(COUNTER_FILE, args.counter_summary)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the forward shards over (batch, head) with no communication "
              "and nothing here uses a second GPU; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    sampler = None
    sample_path = None
    # the board-power sampler is a child process started before this process
    # touches the GPU; the default run records its readings over the timed region
    import shutil
    if args.power_run or (not args.profile_run and not args.no_board and shutil.which("amd-smi")):
        import atexit
        import tempfile
        sample_path = os.path.join(tempfile.mkdtemp(prefix="fp4attn_power_"), "smi.jsonl")
        sampler = start_power_sampler(sample_path)
        atexit.register(_stop_sampler, sampler)
    import torch
    import workloads
    import paper_2609_04105_amd as fa

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.profile_run:
        profile_run(torch, fa)
        return
    if args.power_run:
        try:
            power_run(torch, fa, sampler, sample_path)
        finally:
            _stop_sampler(sampler)
        return

    name = args.workload or workloads.BENCH_WORKLOAD
    w = workloads.WORKLOADS[name]
    q_cpu, k_cpu, v_cpu = workloads.generate(w)
    q, k, v = (t.to(dev) for t in (q_cpu, k_cpu, v_cpu))
    torch.cuda.synchronize()

    ops = fa.quantize_qkv(q, k, v)
    out = torch.empty((w.B, w.H, w.N, w.d), dtype=torch.float32, device=dev)
    bf = (q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16))
    out16 = torch.empty_like(out)

    def fp4_step():
        fa.forward_mxfp4(*ops, softmax_scale=w.softmax_scale, out=out)

    def bf16_step():
        fa.forward_bf16(*bf, softmax_scale=w.softmax_scale, out=out16)

    def quant_step():
        fa.quantize_qkv(q, k, v)

    # warmup (the BF16 kernel warms up in its first timing window)
    for _ in range(args.warmup):
        fp4_step()
    torch.cuda.synchronize()

    # the timed region: exactly `steps` forward steps, synchronized on both sides
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    t_wall0 = time.time()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(args.steps):
        fp4_step()
    ev1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_start) * 1e3
    t_wall1 = time.time()
    fp4_ms = ev0.elapsed_time(ev1) / args.steps

    # the paper's speedup convention: FP4 and BF16 windows interleaved
    pair = {"fp4": fp4_step}
    if not args.no_bf16:
        pair["bf16"] = bf16_step
    _progress(f"timed region: {args.steps} steps, {fp4_ms:.4f} ms per step")
    med, windows = _time_windows(torch, pair, 300.0, args.windows)
    _progress("interleaved FP4 / BF16 windows done")
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
    quantizer = quantizer_roofline(torch, fa, (q, k, v), qms["quant"])
    del ops_anchored, ops8

    flops = w.flops
    tflops = flops / (fp4_ms * 1e-3) / 1e12
    bf16_tflops = flops / (med["bf16"] * 1e-3) / 1e12 if "bf16" in med else None
    c_online = _route_counters("online", name)
    traffic = round(c_online["hbm_bytes"]) if c_online and "hbm_bytes" in c_online else None
    _progress("route and quantizer windows done")
    # the timed kernel back to back on the workload's codes and then on zero codes:
    # its shader clock in steady state, as in the timed region
    cvd = None if args.no_clock_vs_data else clock_vs_data(torch, fa, ops, w, out)
    clk = cvd["workload_codes"]["kernel_clock_ghz"] if cvd else None
    peak_clk = MXFP4_PEAK_TFLOPS * clk / SPEC_CLOCK_GHZ if clk else None
    n_stream = min(stream_blocks(torch), ops[0].numel() // (256 * 64))  # 64 operand bytes per thread
    stream = sustained_mfma_tflops(torch, fa, ops[2].reshape(-1), ops[0].reshape(-1), blocks=n_stream) \
        if n_stream >= 1 else None
    roof = {
        "bound": "mfma",
        "achieved": round(tflops, 2),
        "peak": MXFP4_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(tflops / MXFP4_PEAK_TFLOPS, 4),
        "traffic": traffic,
        "kernel": "fwd_mxfp4_kernel<128, 8, false, 0, 0>",
        "algorithmic_flops_per_launch": flops,
        "algorithmic_bytes_per_launch": int(w.B * w.H * (3 * w.N * w.d * (0.5 + 1 / 32) + 4 * w.N * w.d)),
        "counters": _counter_view(c_online, fp4_ms),
        "measured_clock_ghz": round(clk, 3) if clk else None,
        "peak_at_measured_clock": round(peak_clk, 1) if peak_clk else None,
        "frac_at_measured_clock": round(tflops / peak_clk, 4) if peak_clk else None,
        "sustained_mfma_stream": round(stream, 1) if stream else None,
        "frac_of_sustained_mfma_stream": round(tflops / stream, 4) if stream else None,
        "clock_vs_data": cvd,
    }

    def route(label, ms, route_flops, inputs=name, **extra):
        r = {"ms": round(ms, 5), "tflops": round(route_flops / (ms * 1e-3) / 1e12, 2)}
        r.update(extra)
        r["counters"] = _counter_view(_route_counters(label, inputs), ms)
        return r

    causal_flops = 2.0 * w.d * w.B * w.H * w.N * (w.N + 1)
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
        "fp4_ms_min_interleaved": round(min(windows["fp4"]), 5),
        "bf16_ms_min_interleaved": None if "bf16" not in windows else round(min(windows["bf16"]), 5),
        "interleaved_windows": args.windows,
        "bf16_ms_median_interleaved": None if "bf16" not in med else round(med["bf16"], 5),
        "quantize_qkv_ms": round(qms["quant"], 5),
        "quantizer": quantizer,
        "ex2_pairs_sweep": {str(kx): {"ms": round(med[f"ex2_{kx}"], 5),
                                      "tflops": round(flops / (med[f"ex2_{kx}"] * 1e-3) / 1e12, 2),
                                      "vs_affine": round(med["fp4"] / med[f"ex2_{kx}"], 3),
                                      "counters": _counter_view(_route_counters(f"ex2_{kx}", name),
                                                                med[f"ex2_{kx}"])} for kx in EX2_SWEEP},
        "guard_110_16": route("guard_110_16", med["guard"], flops, vs_online=round(med["fp4"] / med["guard"], 3)),
        "fp8_pv": route("fp8_pv", med["fp8pv"], flops, vs_mxfp4_pv=round(med["fp4"] / med["fp8pv"], 3)),
        # visible (query, key) pairs only: 4 d B H N (N + 1) / 2 flop
        "causal_with_lse": route("causal_lse", med["causal"], causal_flops, flops="4 d B H N (N + 1) / 2"),
        "bf16_counters": None if "bf16" not in med else _counter_view(_route_counters("bf16", name), med["bf16"]),
        "wall_ms_timed_region": round(wall_ms, 3),
        "board": None if sample_path is None else board_readings(sample_path, t_wall0 + 0.2, t_wall1 - 0.2),
        "roofline": roof,
        "gpu": torch.cuda.get_device_name(dev),
        "gfx_target": torch.cuda.get_device_properties(dev).gcnArchName,
        "kernel_source_sha256": _source_sha(),
        "bf16_kernel_source_sha256": _source_sha(BF16_SOURCES),
    }
    del bf, out16
    if not args.no_other_configs and not args.no_bf16 and args.workload is None:
        line["configs"] = other_configs(torch, fa, name)
        _progress("other workloads done")
    if not args.no_paper_shapes and not args.no_bf16:
        line["paper_shapes"] = paper_shape_sweep(torch, fa)
        _progress("paper shapes done")
    if not args.no_cpu_baseline:
        import numpy as np
        line["cpu_baseline"], (rows, o_ref) = cpu_oracle_baseline(w, q_cpu, k_cpu, v_cpu)
        _progress("oracle baseline done")
        # parity of the timed launch on the rows the oracle computed
        fp4_step()
        torch.cuda.synchronize()
        got = out.reshape(-1, w.d)[torch.from_numpy(rows).to(dev)].double().cpu().numpy()
        rel = float(np.linalg.norm(got - o_ref) / np.linalg.norm(o_ref))
        cos = float(np.sum(got * o_ref) / (np.linalg.norm(got) * np.linalg.norm(o_ref)))
        row_rel = np.linalg.norm(got - o_ref, axis=1) / np.linalg.norm(o_ref, axis=1)
        line["parity"] = {"rows": int(len(rows)), "row_set": "the oracle baseline's seeded sampled rows",
                          "o_rel_l2": rel, "o_cos": cos,
                          "o_worst_row_rel_l2": float(row_rel.max()),
                          "gate": {"o_rel_l2_max": 2e-3, "o_cos_min": 0.9999, "o_row_rel_l2_max": 2e-3},
                          "pass": bool(rel <= 2e-3 and cos >= 0.9999 and row_rel.max() <= 2e-3)}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
