"""CPU checks of bench.py's host logic: the route inputs it parses, the
per-route figures it derives from rocprofv3 counter CSVs (written here with
made-up counts whose derived values are known in closed form), and the source
hash that ties a counter file to the kernel it measured.  No GPU is used."""
import csv
import importlib.util
import json
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_host", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_route_inputs_parse(bench):
    assert bench._shape_of("d64_b1h64_n32768")[:4] == (1, 64, 32768, 64)
    B, H, N, d, w = bench._shape_of("long_b1h32_n16384_d128")
    assert (B, H, N, d) == (1, 32, 16384, 128) and w.seed == 4
    with pytest.raises(ValueError):
        bench._shape_of("d64_b1_h64_n32768")
    for label, inputs, family, opts in bench.PROFILE_ROUTES:
        bench._shape_of(inputs)
        assert family in ("fp4", "bf16")
    # causal routes count the visible pairs only
    scores, flop = bench._route_scores("long_b1h32_n16384_d128", {"causal": True})
    assert scores == 32 * 16384 * 16385 / 2 and flop == 4 * 128 * scores


def _write_pass(path, counters_by_dispatch):
    cols = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
            "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
            "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    with open(path, "w", newline="") as f:
        wr = csv.writer(f)
        wr.writerow(cols)
        for disp, (kernel, counters) in enumerate(counters_by_dispatch, start=1):
            for name, val in counters.items():
                # two dimension rows per counter: the summary must add them
                for part in (0.25, 0.75):
                    wr.writerow([disp, disp, "Agent 1", 1, 1, 1, 1024, 7, kernel, 256, 77824, 0, 204, 0, 64, name,
                                 val * part, 0, 1])


def test_counter_summary_derivations(bench, tmp_path):
    routes = [("online", "long_b1h32_n16384_d128", "fp4", {}),
              ("bf16", "d64_b1h64_n32768", "bf16", {})]
    scores0 = 32 * 16384 ** 2
    kib_copy = (256 << 20) / 1024
    fwd0 = "void fp4attn::directp_detail::fwd_mxfp4_kernel<128, 8, false, 0, 0>(fp4attn::directp_detail::KParams)"
    fwd1 = "void fp4attn::(anonymous namespace)::fwd_bf16_kernel<64, 8, false>(BParams)"
    quant = "void fp4attn::quantize_mxfp4_bf16_rows_kernel(...)"
    copy = "__amd_rocclr_copyBuffer"
    p0 = {"SQ_INSTS_VALU": 3.0 * scores0 / 64, "SQ_INSTS_MFMA": 1.0 * scores0 / 64,
          "SQ_INSTS_VALU_TRANS_F32": 0.0, "SQ_VALU_MFMA_BUSY_CYCLES": 0.4 * 1000 * 1024,
          "GRBM_GUI_ACTIVE": 1000 * 8, "SQ_WAVE_CYCLES": 100.0}
    p1 = {"SQ_WAIT_INST_ANY": 25.0, "GRBM_GUI_ACTIVE": 1000 * 8}
    paths = []
    for i, (fwd_counters, copy_counters) in enumerate([
            (p0, {"SQ_INSTS_VALU": 1.0}),
            (p1, {"SQ_WAIT_INST_ANY": 1.0}),
            ({"FETCH_SIZE": 1000.0}, {"FETCH_SIZE": kib_copy / 2}),    # copy reads half: fetch scale 2
            ({"WRITE_SIZE": 500.0}, {"WRITE_SIZE": kib_copy})]):
        path = tmp_path / f"p{i}.csv"
        _write_pass(path, [(copy, copy_counters), (quant, {k: 1.0 for k in fwd_counters}),
                           (fwd0, fwd_counters), (fwd1, fwd_counters)])
        paths.append(str(path))
    out = tmp_path / "counters.json"
    res = bench.counter_summary(str(out), paths, routes=routes)
    assert json.load(open(out)) == json.loads(json.dumps(res))
    r0 = res["routes"][0]
    assert r0["kernel"].startswith("fp4attn::directp_detail::fwd_mxfp4_kernel<128, 8, false, 0, 0>")
    der = r0["derived"]
    assert der["mfma_busy_pct"] == pytest.approx(40.0)
    assert der["valu_non_mfma_per_score"] == pytest.approx(2.0)
    assert der["mfma_per_score"] == pytest.approx(1.0)
    assert der["trans_per_score"] == 0.0
    assert der["wait_inst_any_pct_of_wave_cycles"] == pytest.approx(25.0)
    assert der["fetch_bytes"] == pytest.approx(1000 * 1024 * 2) and der["write_bytes"] == pytest.approx(500 * 1024)
    assert der["algorithmic_bytes"] == pytest.approx(32 * (3 * 16384 * 128 * (0.5 + 1 / 32) + 4 * 16384 * 128))
    assert r0["source_sha256"] == bench._source_sha()
    r1 = res["routes"][1]
    assert r1["family"] == "bf16" and r1["derived"]["algorithmic_bytes"] == 64 * 10 * 32768 * 64
    assert r1["source_sha256"] == bench._source_sha(bench.BF16_SOURCES)


def test_counter_summary_refuses_a_route_count_mismatch(bench, tmp_path):
    path = tmp_path / "p.csv"
    _write_pass(path, [("__amd_rocclr_copyBuffer", {"FETCH_SIZE": 1.0})])
    with pytest.raises(SystemExit):
        bench.counter_summary(str(tmp_path / "o.json"), [str(path)], routes=bench.PROFILE_ROUTES)


def test_source_hash_ignores_comments(bench, tmp_path):
    a, b = tmp_path / "a.hip", tmp_path / "b.hip"
    a.write_text("int x = 1;  // one\n\n// note\nint y;\n")
    b.write_text("int x = 1;\nint y;  // another comment\n")
    assert bench._source_sha([str(a)]) == bench._source_sha([str(b)])
    b.write_text("int x = 2;\nint y;\n")
    assert bench._source_sha([str(a)]) != bench._source_sha([str(b)])
