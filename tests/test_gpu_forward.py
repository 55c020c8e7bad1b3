"""GPU parity of the Direct-P MXFP4 forward against the oracle.

Gates: Direct-P code mismatch fraction <= 1e-4, output relative L2 <= 2e-3
and cosine >= 0.9999; all rows for the small workloads,
4096 sampled rows (the same launch as the timed forward) for the large ones.
"""
import numpy as np
import pytest
import torch

import workloads
from parity import (check_directp_dump, check_fp8_dump, check_guarded_dump, check_output, gpu_operands, load_workload,
                    oracle_rows, oracle_rows_two_maps, unpack_codes)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fa():
    import paper_2609_04105_amd as fa
    return fa


def _run_and_check(fa, host64, dev, rows, label, softmax_scale=None, affine=(1.5, 1.2), ex2_pairs=None,
                   causal=False, lse=False):
    q, k, v = host64
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d) if softmax_scale is None else softmax_scale
    ops = gpu_operands(*dev)
    row_ids = torch.from_numpy(np.asarray(rows, dtype=np.int64)).cuda()
    print(f"[{label}] B{B} H{H} N{N} d{d} rows={len(rows)} ex2_pairs={ex2_pairs} causal={causal}", flush=True)
    dump = fa.debug_directp_mxfp4(*ops, row_ids, softmax_scale=s, affine_a=affine[0], affine_b=affine[1],
                                  ex2_pairs=ex2_pairs or 0, causal=causal, lse=lse)
    lse_out = torch.empty((B, H, N), dtype=torch.float32, device="cuda") if lse else None
    out = fa.forward_mxfp4(*ops, softmax_scale=s, affine_a=affine[0], affine_b=affine[1], ex2_pairs=ex2_pairs,
                           causal=causal, lse=lse_out)
    torch.cuda.synchronize()
    # the test hook runs the same kernel: identical output
    assert torch.equal(out, dump["out"]), f"{label}: debug launch output differs from the forward"
    ref = oracle_rows(q, k, v, rows, s, *affine, ex2_pairs=ex2_pairs or 0, causal=causal)
    if lse:
        assert torch.equal(lse_out, dump["lse"])
        got_lse = lse_out.reshape(-1)[row_ids].cpu().numpy().astype(np.float64)
        err = np.abs(got_lse - ref["LSE"])
        print(f"[{label}] LSE max abs error {err.max():.2e}", flush=True)
        assert np.all(err <= 1e-4 + 1e-6 * np.abs(ref["LSE"])), f"{label}: LSE error {err.max()}" 
    mismatch = check_directp_dump(dump, ref, label)
    print(f"[{label}] code mismatch {mismatch:.2e}", flush=True)
    got = out.reshape(-1, d)[torch.from_numpy(np.asarray(rows)).cuda()].cpu().numpy()
    check_output(got, ref["O"], label)
    return out, ops


def test_tiny_all_rows(fa):
    host64, dev = load_workload("tiny_b1h1_n128_d64")
    _run_and_check(fa, host64, dev, workloads.sampled_rows("tiny_b1h1_n128_d64"), "tiny")


def test_small_all_rows(fa):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    _run_and_check(fa, host64, dev, workloads.sampled_rows("small_b1h8_n1024_d64"), "small")


@pytest.mark.parametrize("N,d", [(384, 128), (640, 64), (1152, 128)])
def test_ragged_tiles_all_rows(fa, N, d):
    """Several key tiles and a query-tile count that does not fill whole 8-wave groups."""
    g = torch.Generator().manual_seed(N + d)
    q, k, v = (torch.randn(1, 2, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    _run_and_check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(2 * N), f"ragged N{N} d{d}")


def test_wide_launch_sampled(fa):
    """The 8-wave (256-row) workgroup path at a size the oracle checks on every 7th row."""
    g = torch.Generator().manual_seed(7)
    B, H, N, d = 1, 128, 512, 128
    q, k, v = (torch.randn(B, H, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    _run_and_check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(0, B * H * N, 7), "wide")


def test_wide_launch_two_tiles(fa):
    """The 8-wave path with two key tiles per head: the tile fetches run three tiles
    ahead, so most of them read past the head's last key (zeros, never used)."""
    g = torch.Generator().manual_seed(8)
    B, H, N, d = 1, 256, 256, 128
    q, k, v = (torch.randn(B, H, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    _run_and_check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(0, B * H * N, 5), "wide two tiles")


@pytest.mark.parametrize("H,d", [(24, 64), (24, 128), (36, 64)])
def test_half_round_tail_launch(fa, H, d):
    """B1 N4096 grids whose eight-wave launch would end in a mostly empty round, so
    the launch takes four-wave workgroups: H24 (384 eight-wave workgroups, two
    rounds, the second half empty) and H36 d64 (576, a third round a quarter
    full: 1152 four-wave workgroups); every 23rd row checked."""
    g = torch.Generator().manual_seed(9)
    B, N = 1, 4096
    q, k, v = (torch.randn(B, H, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    _run_and_check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(0, B * H * N, 23), f"tail H{H} d{d}")


@pytest.mark.parametrize("name", ["small_b1h8_n1024_d64", "outlier_b2h16_n4096_d128", "student_t_b1h32_n8192_d128",
                                  "long_b1h32_n16384_d128"])
def test_codes_against_plain_fp64_map(fa, name):
    """The GPU's Direct-P codes and block exponents against the code map of eq.
    affine-code-map written out in fp64 (the oracle's ``affine64`` mode: y = z log2 e,
    E_B = floor(max y), q = Q_E2M1(max(0, A (y - E_B + log2 6) + B)), no fp32
    folding of the coefficients), at the same 1e-4 gate; all rows of the small
    workload, the 4096 sampled rows of the outlier, Student-t and long ones.  The output is held to the
    fp64 map's output too.  Both mismatch fractions are printed: against the fp64
    map and against the oracle's fp32 fused multiply-add decision."""
    (q, k, v), dev = load_workload(name)
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d)
    rows = workloads.sampled_rows(name)
    ops = gpu_operands(*dev)
    row_ids = torch.from_numpy(np.asarray(rows, dtype=np.int64)).cuda()
    print(f"[{name}] plain fp64 map: B{B} H{H} N{N} d{d} rows={len(rows)}", flush=True)
    dump = fa.debug_directp_mxfp4(*ops, row_ids, softmax_scale=s)
    torch.cuda.synchronize()
    got_codes = unpack_codes(dump["p_codes"].cpu().numpy()) & 7
    got_E = dump["block_exp"].cpu().numpy().astype(np.int64)
    got_O = dump["out"].reshape(-1, d)[row_ids].cpu().numpy()
    del dump, ops
    ref = oracle_rows_two_maps(q, k, v, rows, s)
    frac = {}
    for mode, tag in (("affine64", "64"), ("affine32", "32")):
        bad = got_codes != ref["codes" + tag]
        frac[mode] = (float(np.mean(bad)), float(np.mean(got_E != ref["E" + tag])))
        print(f"[{name}] vs {mode}: code mismatch {frac[mode][0]:.3e} ({int(bad.sum())} of {bad.size}), "
              f"block exponent mismatch {frac[mode][1]:.3e}", flush=True)
    check_output(got_O, ref["O64"], f"{name} vs affine64")
    assert frac["affine64"][0] <= 1e-4 and frac["affine64"][1] <= 1e-4, frac


@pytest.mark.parametrize("name", ["outlier_b2h16_n4096_d128", "student_t_b1h32_n8192_d128",
                                  "long_b1h32_n16384_d128"])
def test_full_size_sampled_rows(fa, name):
    host64, dev = load_workload(name)
    _run_and_check(fa, host64, dev, workloads.sampled_rows(name), name)


def _check_byte_operands(fa, ops_cpu, rows, label, causal=False, guard=None, pv_fp8=False):
    """Forward and Direct-P dump of MXFP4 operand bytes against the oracle on the
    flattened query ``rows`` (the same bytes feed both sides; with ``guard`` the
    key order of the bytes is the anchor order)."""
    from oracle import directp, fp8pv
    from oracle import guard as guard_oracle
    B, H, N, half_d = ops_cpu[0].shape
    d = 2 * half_d
    s = 1.0 / np.sqrt(d)
    rows = np.asarray(rows, dtype=np.int64)
    print(f"[{label}] B{B} H{H} N{N} d{d} rows={len(rows)}: GPU launches", flush=True)
    ops = tuple(t.cuda() for t in ops_cpu)
    row_ids = torch.from_numpy(rows).cuda()
    dump = fa.debug_directp_mxfp4(*ops, row_ids, softmax_scale=s, causal=causal, guard=guard, pv_fp8=pv_fp8)
    out = fa.forward_mxfp4(*ops, softmax_scale=s, causal=causal, guard=guard, pv_fp8=pv_fp8)
    torch.cuda.synchronize()
    assert torch.equal(out, dump["out"]), f"{label}: debug launch output differs from the forward"
    assert bool(torch.isfinite(out).all()), f"{label}: non-finite output"
    got = out.reshape(-1, d)[row_ids].cpu().numpy()
    del ops, out
    dump = {key: val for key, val in dump.items() if key != "out"}
    print(f"[{label}] oracle", flush=True)
    keys = ("O", "ebar", "D", "codes") if guard else ("O", "E", "M", "D", "codes")
    ref = {key: [] for key in keys}
    order = []
    for bh in np.unique(rows // N):
        b, h = divmod(int(bh), H)
        sel = np.nonzero(rows // N == bh)[0]
        head = [t[b, h].numpy() for t in ops_cpu]
        if guard:
            res = guard_oracle.forward_rows(*head, rows[sel] % N, s, *guard)
        elif pv_fp8:
            res = fp8pv.forward_rows(*head, rows[sel] % N, s, causal=causal)
        else:
            res = directp.forward_rows(*head, rows[sel] % N, s, causal=causal)
        for key in ref:
            ref[key].append(res[key])
        order.append(sel)
    order = np.concatenate(order)
    ref = {key: np.concatenate(val)[np.argsort(order)] for key, val in ref.items()}
    if guard:
        mismatch = check_guarded_dump(dump, ref, label)
    elif pv_fp8:
        mismatch = check_fp8_dump(dump, ref, label)
    else:
        mismatch = check_directp_dump(dump, ref, label)
    print(f"[{label}] code mismatch {mismatch:.2e}", flush=True)
    check_output(got, ref["O"], label)


@pytest.mark.parametrize("d,causal", [(128, False), (128, True), (64, False), (64, True)])
def test_longest_sequence_sampled_rows(fa, d, causal):
    """N = 2^22 keys, the largest the entry point accepts: every byte offset within
    the head near its 32-bit limit, 32768 key tiles per workgroup; d = 64 takes
    128-query workgroups at four waves per SIMD (one-step pipeline).  Rows: the first and last of the
    sequence, of a query tile and of a workgroup, and random ones."""
    N = 1 << 22
    ops_cpu = workloads.random_mxfp4_operands(1, 1, N, d, seed=22 + d)
    rows = np.unique(np.concatenate([[0, 1, 127, 128, 255, 256, N // 2 + 31, N - 257, N - 256, N - 129, N - 128,
                                      N - 1], np.random.default_rng(22).integers(0, N, 8)]))
    _check_byte_operands(fa, ops_cpu, rows, f"N=2^22 d{d} causal={causal}", causal=causal)


@pytest.mark.parametrize("route", ["guard_110_16", "fp8_pv"])
def test_longest_sequence_other_routes(fa, route):
    """N = 2^22 on the sampled guard (the paper's margin and shift; the bytes'
    first 128 keys are the anchors) and on the FP8 P/V route (Vt 2^22 bytes per
    row of d)."""
    N = 1 << 22
    pv_fp8 = route == "fp8_pv"
    ops_cpu = workloads.random_mxfp4_operands(1, 1, N, 128, seed=23, v_fp8=pv_fp8)
    rows = np.unique(np.concatenate([[0, 1, 255, 256, N // 2 + 31, N - 257, N - 256, N - 1],
                                     np.random.default_rng(23).integers(0, N, 8)]))
    _check_byte_operands(fa, ops_cpu, rows, f"N=2^22 {route}", guard=None if pv_fp8 else (110, 16), pv_fp8=pv_fp8)


def test_largest_grid_sampled_rows(fa):
    """More than 2^16 (batch, head) slices in one launch; rows of the first, the
    last and random slices."""
    B, H, N = 2, 32775, 256
    ops_cpu = workloads.random_mxfp4_operands(B, H, N, 64, seed=16)
    rng = np.random.default_rng(16)
    heads = np.unique(np.concatenate([[0, 1, H - 1, H, B * H - 2, B * H - 1], rng.integers(0, B * H, 10)]))
    rows = np.unique(np.concatenate([bh * N + np.array([0, 1, 127, 128, N - 1]) for bh in heads]))
    _check_byte_operands(fa, ops_cpu, rows, f"B{B} H{H}")


def test_concurrent_threads_and_streams(fa):
    """No state is shared between calls: two host threads, each enqueueing
    forwards on its own stream (default priority), reproduce the sequential
    outputs bit for bit."""
    import threading
    g = torch.Generator().manual_seed(31)
    shapes = [(1, 4, 1024, 128), (2, 3, 512, 64)]
    cases = []
    for shape in shapes:
        q, k, v = (torch.randn(*shape, generator=g).to(torch.bfloat16).cuda() for _ in range(3))
        ops = fa.quantize_qkv(q, k, v)
        cases.append((ops, fa.forward_mxfp4(*ops), fa.forward_mxfp4(*ops, causal=True)))
    torch.cuda.synchronize()
    results, errors = {}, []

    def worker(i):
        try:
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                ops = cases[i][0]
                outs = [(fa.forward_mxfp4(*ops), fa.forward_mxfp4(*ops, causal=True)) for _ in range(4)]
            stream.synchronize()
            results[i] = outs
        except Exception as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(cases))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for i, (_, ref, ref_causal) in enumerate(cases):
        for out, out_causal in results[i]:
            assert torch.equal(out, ref) and torch.equal(out_causal, ref_causal)


def test_affine_variant_and_scale(fa):
    """The Wan fit (A, B) = (1.6, 0.95) and a non-default softmax scale."""
    host64, dev = load_workload("small_b1h8_n1024_d64", H=2)
    _run_and_check(fa, host64, dev, np.arange(2 * 1024), "wan affine", softmax_scale=0.2, affine=(1.6, 0.95))


def test_affine_variant_long_sampled_rows(fa):
    """The Wan fit on the long workload's 4096 sampled rows (the timed launch shape)."""
    name = "long_b1h32_n16384_d128"
    host64, dev = load_workload(name)
    _run_and_check(fa, host64, dev, workloads.sampled_rows(name), f"{name} wan affine", affine=(1.6, 0.95))


def test_extreme_logits_stay_finite(fa):
    """Rows whose log2 range exceeds the E8M0 byte range (zero blocks, reference jumps)."""
    g = torch.Generator().manual_seed(11)
    N, d = 1024, 128
    q, k, v = (torch.randn(1, 1, N, d, generator=g) for _ in range(3))
    q[..., :4] *= 30.0
    k[..., :4] *= 30.0
    q, k, v = (t.to(torch.bfloat16) for t in (q, k, v))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    out, _ = _run_and_check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(N), "extreme")
    assert torch.isfinite(out).all()


@pytest.mark.parametrize("case", ["q_zero", "v_zero", "v_pow2"])
def test_degenerate_inputs(fa, case):
    """Degenerate inputs of the method, on a launch of several tiles.  Q = 0: every
    score is 0, so every block has E_B = 0 and one code everywhere, and O is the
    mean of the represented V rows.  V = 0: O = 0 exactly.  V = 2^-3 everywhere:
    every V block is represented exactly, so O = 2^-3 up to fp32 summation."""
    g = torch.Generator().manual_seed(12)
    B, H, N, d = 1, 2, 640, 128
    q, k, v = (torch.randn(B, H, N, d, generator=g) for _ in range(3))
    if case == "q_zero":
        q.zero_()
    elif case == "v_zero":
        v.zero_()
    else:
        v.fill_(0.125)
    q, k, v = (t.to(torch.bfloat16) for t in (q, k, v))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    rows = np.arange(B * H * N)
    print(f"[degenerate {case}] B{B} H{H} N{N} d{d}", flush=True)
    ops = gpu_operands(q.cuda(), k.cuda(), v.cuda())
    dump = fa.debug_directp_mxfp4(*ops, torch.from_numpy(rows).cuda())
    out = fa.forward_mxfp4(*ops)
    torch.cuda.synchronize()
    assert torch.equal(out, dump["out"])
    ref = oracle_rows(*host64, rows, 1.0 / np.sqrt(d))
    mismatch = check_directp_dump(dump, ref, case)
    got = out.reshape(-1, d).cpu().numpy().astype(np.float64)
    assert np.isfinite(got).all()
    if case == "q_zero":
        assert np.all(ref["E"] == 0) and np.all(ref["codes"] == ref["codes"][0, 0])
        vhat = np.stack([fa_oracle_vhat(host64[2][0, h]) for h in range(H)])      # [H, N, d]
        mean = vhat.mean(axis=1)                                                 # [H, d]
        np.testing.assert_allclose(got.reshape(H, N, d), np.broadcast_to(mean[:, None], (H, N, d)),
                                   rtol=1e-5, atol=2e-6)
    elif case == "v_zero":
        assert np.all(got == 0.0)
    else:
        np.testing.assert_allclose(got, 0.125, rtol=1e-5, atol=0)
    if case != "v_zero":
        check_output(got, ref["O"], case)
    print(f"[degenerate {case}] code mismatch {mismatch:.2e}", flush=True)


def fa_oracle_vhat(v):
    """Represented V̂ [N, d] of one head: the oracle's MXFP4 quantization along
    the sequence, decoded."""
    from oracle import mxfp4
    codes, scales = mxfp4.quantize(v, axis=-2)          # stored transposed: [d, N]
    return mxfp4.dequantize(codes, scales).T


def test_deterministic_and_fully_overwritten(fa):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    ops = gpu_operands(*dev)
    out1 = torch.full((1, 8, 1024, 64), float("nan"), device="cuda")
    fa.forward_mxfp4(*ops, out=out1)
    out2 = torch.full_like(out1, float("nan"))
    fa.forward_mxfp4(*ops, out=out2)
    torch.cuda.synchronize()
    assert torch.isfinite(out1).all()
    assert torch.equal(out1, out2)


def test_bf16_output_is_rounded_fp32_output(fa):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    ops = gpu_operands(*dev)
    o32 = fa.forward_mxfp4(*ops)
    o16 = fa.forward_mxfp4(*ops, out_dtype=torch.bfloat16)
    assert torch.equal(o16, o32.to(torch.bfloat16))


def test_error_paths_do_not_launch(fa):
    host64, dev = load_workload("tiny_b1h1_n128_d64")
    ops = gpu_operands(*dev)
    out = torch.full((1, 1, 128, 64), 7.0, device="cuda")
    lib = fa.lib
    import ctypes
    p = [ctypes.c_void_p(t.data_ptr()) for t in ops]
    o = ctypes.c_void_p(out.data_ptr())
    assert lib.fp4attn_forward_mxfp4(*p, 1, 1, 96, 64, 0.125, 1.5, 1.2, o, 0, None) == 1   # N not /128
    assert lib.fp4attn_forward_mxfp4(*p, 1, 1, 128, 96, 0.125, 1.5, 1.2, o, 0, None) == 2  # d unsupported
    assert lib.fp4attn_forward_mxfp4(*p, 1, 1, 128, 64, -1.0, 1.5, 1.2, o, 0, None) == 1   # bad scale
    assert lib.fp4attn_forward_mxfp4(*p, 1, 1, 128, 64, 0.125, 0.0, 1.2, o, 0, None) == 1  # bad A
    assert lib.fp4attn_forward_mxfp4(*p, 1, 1, 128, 64, 0.125, 1.5, 1.2, o, 5, None) == 1  # bad dtype
    bad = ctypes.c_void_p(out.data_ptr() + 4)
    assert lib.fp4attn_forward_mxfp4(*p, 1, 1, 128, 64, 0.125, 1.5, 1.2, bad, 0, None) == 1  # misaligned
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
    with pytest.raises(fa.Fp4AttnError):
        fa.forward_mxfp4(*ops, softmax_scale=float("inf"))


@pytest.mark.parametrize("n_dump", [0, 1])
# (1, 24, 4096, 128): 384 eight-wave workgroups would leave a half-empty second
# round, so the launch takes 768 four-wave ones
# (1, 36, 4096, 64): 576 eight-wave workgroups, a third round a quarter full: 1152
# four-wave ones; (1, 32, 4096, 128): 512, two full rounds: eight waves
@pytest.mark.parametrize("B,H,N,d,wgs", [(1, 2, 384, 128, 6), (1, 128, 512, 128, 256), (1, 24, 4096, 128, 768),
                                         (1, 36, 4096, 64, 1152), (1, 32, 4096, 128, 512)])
def test_workgroup_clock_record(fa, B, H, N, d, wgs, n_dump):
    """The test entry point's per-workgroup clock record, with and without rows to
    dump: exactly the launch's workgroups write it, with a plausible shader clock,
    and the output equals the forward's."""
    g = torch.Generator().manual_seed(11)
    q, k, v = (torch.randn(B, H, N, d, generator=g).to(torch.bfloat16).cuda() for _ in range(3))
    ops = gpu_operands(q, k, v)
    print(f"[clock] B{B} H{H} N{N} d{d} dump rows {n_dump}", flush=True)
    r = fa.debug_directp_mxfp4(*ops, torch.zeros(n_dump, dtype=torch.int64, device="cuda"), wg_clock=True)
    out = fa.forward_mxfp4(*ops)
    torch.cuda.synchronize()
    assert torch.equal(out, r["out"])
    c = r["wg_clock"].cpu()
    assert c.shape == (B * H * N // 128, 2)
    assert bool((c[:wgs] > 0).all()) and bool((c[wgs:] == 0).all())
    ghz = float(c[:, 0].sum()) / (float(c[:, 1].sum()) / 100e6) / 1e9
    print(f"[clock] {ghz:.3f} GHz", flush=True)
    assert 0.3 < ghz < 3.0


@pytest.mark.parametrize("ex2_pairs", [1, 2, 4, 8, 16])
def test_ex2_mixing_small_all_rows(fa, ex2_pairs):
    """Native-exponential pair mixing against the oracle's fp32 decision (the
    hardware exponential may move a value across an E2M1 boundary only within
    its last bits, inside the 1e-4 code-mismatch gate)."""
    host64, dev = load_workload("small_b1h8_n1024_d64")
    _run_and_check(fa, host64, dev, workloads.sampled_rows("small_b1h8_n1024_d64"), f"small ex2={ex2_pairs}",
                   ex2_pairs=ex2_pairs)


@pytest.mark.parametrize("name,ex2_pairs", [("long_b1h32_n16384_d128", 4), ("long_b1h32_n16384_d128", 16),
                                            ("outlier_b2h16_n4096_d128", 4), ("student_t_b1h32_n8192_d128", 4)])
def test_ex2_mixing_large_sampled_rows(fa, name, ex2_pairs):
    host64, dev = load_workload(name)
    _run_and_check(fa, host64, dev, workloads.sampled_rows(name), f"{name} ex2={ex2_pairs}", ex2_pairs=ex2_pairs)


def test_extended_entry_with_defaults_is_the_plain_forward(fa):
    host64, dev = load_workload("outlier_b2h16_n4096_d128")
    ops = gpu_operands(*dev)
    a = fa.forward_mxfp4(*ops)
    b = fa.forward_mxfp4(*ops, ex2_pairs=0)
    c = fa.forward_mxfp4(*ops, out_dtype=torch.bfloat16, ex2_pairs=0)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert torch.equal(c, a.to(torch.bfloat16))


def test_ex2_density_fidelity_against_exact_attention(fa):
    """Operator error of each density against exact attention on the unquantized
    inputs (Sec. "Metrics": cosine, relative L2, RMSE), 4096 sampled rows of the
    long workload: more native-exponential pairs, lower error, as in the paper's
    density sweep (Table b300-tuning)."""
    from oracle import exact
    name = "long_b1h32_n16384_d128"
    (q, k, v), dev = load_workload(name)
    ops = gpu_operands(*dev)
    rows = workloads.sampled_rows(name)
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d)
    ref = np.zeros((len(rows), d))
    for bh in np.unique(rows // N):
        sel = np.nonzero(rows // N == bh)[0]
        b, h = divmod(int(bh), H)
        ref[sel] = exact.attention(q[b, h][rows[sel] % N], k[b, h], v[b, h], s)
    idx = torch.from_numpy(rows).cuda()
    rels = []
    for kx in (0, 1, 2, 4, 16):
        out = fa.forward_mxfp4(*ops, ex2_pairs=kx)
        got = out.reshape(-1, d)[idx].cpu().numpy()
        cos, rel, rmse = exact.error_metrics(got, ref)
        print(f"[fidelity] ex2_pairs={kx:2d} cos {cos:.6f} rel-L2 {rel:.6f} RMSE {rmse:.6f}", flush=True)
        rels.append(rel)
    assert all(a > b for a, b in zip(rels, rels[1:])), rels


# ---- sampled QK guard (Alg. 3) ------------------------------------------------------------

def _run_guarded(fa, host64, dev, rows, label, margin, shift, ex2_pairs=0, softmax_scale=None):
    from parity import check_guarded_dump, oracle_rows_guarded
    q, k, v = host64
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d) if softmax_scale is None else softmax_scale
    ops = fa.quantize_qkv(*dev, anchored=True)
    row_ids = torch.from_numpy(np.asarray(rows, dtype=np.int64)).cuda()
    print(f"[{label}] guard M={margin} L={shift} ex2={ex2_pairs} B{B} H{H} N{N} d{d} rows={len(rows)}", flush=True)
    dump = fa.debug_directp_mxfp4(*ops, row_ids, softmax_scale=s, ex2_pairs=ex2_pairs, guard=(margin, shift))
    out = fa.forward_mxfp4(*ops, softmax_scale=s, ex2_pairs=ex2_pairs, guard=(margin, shift))
    torch.cuda.synchronize()
    assert torch.equal(out, dump["out"])
    ref = oracle_rows_guarded(q, k, v, rows, s, margin, shift, ex2_pairs)
    mismatch = check_guarded_dump(dump, ref, label)
    got = out.reshape(-1, d)[torch.from_numpy(np.asarray(rows)).cuda()].cpu().numpy()
    assert np.all(np.isfinite(got))
    print(f"[{label}] code mismatch {mismatch:.2e}", flush=True)
    check_output(got, ref["O"], label)


@pytest.mark.parametrize("margin,shift", [(8, 0), (20, 16), (110, 16), (112, 14)])
def test_guard_small_all_rows(fa, margin, shift):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    _run_guarded(fa, host64, dev, workloads.sampled_rows("small_b1h8_n1024_d64"), "small", margin, shift)


@pytest.mark.parametrize("ex2_pairs", [4, 16])
def test_guard_with_native_exponential_pairs(fa, ex2_pairs):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    _run_guarded(fa, host64, dev, workloads.sampled_rows("small_b1h8_n1024_d64"), "small", 110, 16, ex2_pairs)


@pytest.mark.parametrize("name", ["outlier_b2h16_n4096_d128", "student_t_b1h32_n8192_d128", "long_b1h32_n16384_d128"])
def test_guard_full_size_sampled_rows(fa, name):
    host64, dev = load_workload(name)
    _run_guarded(fa, host64, dev, workloads.sampled_rows(name), name, 110, 16)


def test_guard_tiny_and_ragged(fa):
    host64, dev = load_workload("tiny_b1h1_n128_d64")
    _run_guarded(fa, host64, dev, np.arange(128), "tiny", 110, 16)
    g = torch.Generator().manual_seed(33)
    q, k, v = (torch.randn(1, 2, 1152, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    _run_guarded(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(2 * 1152), "ragged N1152", 20, 16)


def test_guard_extreme_logits(fa):
    """Logits in the thousands (the regime the guard serves): finite output that
    matches the oracle."""
    g = torch.Generator().manual_seed(34)
    q = (torch.randn(1, 2, 512, 64, generator=g) * 60).to(torch.bfloat16)
    k = (torch.randn(1, 2, 512, 64, generator=g) * 4).to(torch.bfloat16)
    v = torch.randn(1, 2, 512, 64, generator=g).to(torch.bfloat16)
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    _run_guarded(fa, host64, (q.cuda(), k.cuda(), v.cuda()), np.arange(1024), "extreme", 110, 16)


def test_guard_fidelity_against_exact_attention(fa):
    """Operator error of the guarded route against exact attention (4096 sampled rows
    of the long workload): with a small margin it equals the online route's; the
    paper's (110, 16) floors sub-anchor blocks of these flat Gaussian rows."""
    from oracle import exact
    name = "long_b1h32_n16384_d128"
    (q, k, v), dev = load_workload(name)
    rows = workloads.sampled_rows(name)
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d)
    ref = np.zeros((len(rows), d))
    for bh in np.unique(rows // N):
        sel = np.nonzero(rows // N == bh)[0]
        b, h = divmod(int(bh), H)
        ref[sel] = exact.attention(q[b, h][rows[sel] % N], k[b, h], v[b, h], s)
    idx = torch.from_numpy(rows).cuda()
    online = fa.forward_mxfp4(*gpu_operands(*dev)).reshape(-1, d)[idx].cpu().numpy()
    anch = fa.quantize_qkv(*dev, anchored=True)
    rel = {"online": exact.error_metrics(online, ref)[1]}
    for ml in ((8, 0), (110, 16)):
        got = fa.forward_mxfp4(*anch, guard=ml).reshape(-1, d)[idx].cpu().numpy()
        cos, rel[ml], rmse = exact.error_metrics(got, ref)
        print(f"[fidelity] guard M={ml[0]} L={ml[1]}: cos {cos:.6f} rel-L2 {rel[ml]:.6f} RMSE {rmse:.6f}", flush=True)
    print(f"[fidelity] online reference: rel-L2 {rel['online']:.6f}", flush=True)
    assert abs(rel[(8, 0)] / rel["online"] - 1) < 0.05



# ---- causal forward and the saved row normaliser ------------------------------------------

@pytest.mark.parametrize("ex2_pairs", [0, 4, 16])
def test_causal_small_all_rows(fa, ex2_pairs):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    _run_and_check(fa, host64, dev, workloads.sampled_rows("small_b1h8_n1024_d64"), f"causal small ex2={ex2_pairs}",
                   ex2_pairs=ex2_pairs, causal=True, lse=True)


@pytest.mark.parametrize("N,d,H", [(128, 64, 1), (384, 128, 2), (1152, 128, 2), (512, 128, 128)])
def test_causal_tiles_all_rows(fa, N, d, H):
    """One key tile, 4-wave workgroups with a partial last group, and the 8-wave launch."""
    g = torch.Generator().manual_seed(N + d + H)
    q, k, v = (torch.randn(1, H, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    rows = np.arange(H * N) if H * N <= 4096 else np.arange(0, H * N, 11)
    _run_and_check(fa, host64, (q.cuda(), k.cuda(), v.cuda()), rows, f"causal N{N} d{d} H{H}", causal=True, lse=True)


@pytest.mark.parametrize("name", ["outlier_b2h16_n4096_d128", "student_t_b1h32_n8192_d128", "long_b1h32_n16384_d128"])
def test_causal_large_sampled_rows(fa, name):
    host64, dev = load_workload(name)
    _run_and_check(fa, host64, dev, workloads.sampled_rows(name), f"causal {name}", causal=True, lse=True)


def test_lse_noncausal_and_guarded(fa):
    host64, dev = load_workload("outlier_b2h16_n4096_d128")
    rows = workloads.sampled_rows("outlier_b2h16_n4096_d128")
    _run_and_check(fa, host64, dev, rows, "lse outlier", lse=True)
    from parity import oracle_rows_guarded
    q, k, v = host64
    B, H, N, d = q.shape
    ops = fa.quantize_qkv(*dev, anchored=True)
    lse = torch.empty((B, H, N), dtype=torch.float32, device="cuda")
    fa.forward_mxfp4(*ops, guard=(110, 16), lse=lse)
    ref = oracle_rows_guarded(q, k, v, rows, 1 / np.sqrt(d), 110, 16)
    err = np.abs(lse.reshape(-1)[torch.from_numpy(rows).cuda()].cpu().numpy() - ref["LSE"])
    print(f"[lse guard] max abs error {err.max():.2e}", flush=True)
    assert np.all(err <= 1e-4 + 1e-6 * np.abs(ref["LSE"]))


def test_causal_first_rows_see_only_their_prefix(fa):
    """Row 0 attends to key 0 alone: O_0 is V_0's represented value (up to the
    epilogue's fp32 division), and changing keys after a row leaves that row's
    output bit-identical."""
    g = torch.Generator().manual_seed(5)
    q, k, v = (torch.randn(1, 1, 512, 64, generator=g).to(torch.bfloat16) for _ in range(3))
    ops = gpu_operands(q.cuda(), k.cuda(), v.cuda())
    o1 = fa.forward_mxfp4(*ops, causal=True)
    k2, v2 = k.clone(), v.clone()
    k2[:, :, 300:] = torch.randn(1, 1, 212, 64, generator=g).to(torch.bfloat16)
    v2[:, :, 300:] = torch.randn(1, 1, 212, 64, generator=g).to(torch.bfloat16)
    ops2 = gpu_operands(q.cuda(), k2.cuda(), v2.cuda())
    o2 = fa.forward_mxfp4(*ops2, causal=True)
    torch.cuda.synchronize()
    # keys 300.. share V blocks with keys 288..299 (blocks of 32 along the sequence), so rows
    # below 288 are untouched
    assert torch.equal(o1[:, :, :288], o2[:, :, :288])
    from oracle import mxfp4
    vc, vs = mxfp4.quantize(workloads.as_f64(v)[0, 0], axis=-2)
    v_hat = mxfp4.scaled_operand(vc, vs).T[0] / 6.0
    np.testing.assert_allclose(o1[0, 0, 0].cpu().numpy().astype(np.float64), v_hat, rtol=3e-7, atol=0)


# ---- FP8 (E4M3) P and V -----------------------------------------------------------------

def _run_fp8(fa, host64, dev, rows, label, causal=False):
    from parity import check_fp8_dump, oracle_rows_fp8
    q, k, v = host64
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d)
    ops = fa.quantize_qkv(*dev, pv_fp8=True)
    row_ids = torch.from_numpy(np.asarray(rows, dtype=np.int64)).cuda()
    print(f"[{label}] fp8 P/V causal={causal} B{B} H{H} N{N} d{d} rows={len(rows)}", flush=True)
    dump = fa.debug_directp_mxfp4(*ops, row_ids, softmax_scale=s, pv_fp8=True, causal=causal, lse=True)
    lse = torch.empty((B, H, N), dtype=torch.float32, device="cuda")
    out = fa.forward_mxfp4(*ops, softmax_scale=s, pv_fp8=True, causal=causal, lse=lse)
    torch.cuda.synchronize()
    assert torch.equal(out, dump["out"]) and torch.equal(lse, dump["lse"])
    ref = oracle_rows_fp8(q, k, v, rows, s, causal)
    mismatch = check_fp8_dump(dump, ref, label)
    got = out.reshape(-1, d)[row_ids].cpu().numpy()
    err = np.abs(lse.reshape(-1)[row_ids].cpu().numpy() - ref["LSE"])
    print(f"[{label}] payload mismatch {mismatch:.2e}  LSE err {err.max():.2e}", flush=True)
    check_output(got, ref["O"], label)
    # ln of the denominator: the same fp32 summation bound as the denominator itself
    assert np.all(err <= max(1e-4, N * 2.0 ** -24) + 1e-6 * np.abs(ref["LSE"]))


@pytest.mark.parametrize("causal", [False, True])
def test_fp8pv_small_all_rows(fa, causal):
    host64, dev = load_workload("small_b1h8_n1024_d64")
    _run_fp8(fa, host64, dev, workloads.sampled_rows("small_b1h8_n1024_d64"), "small", causal)


@pytest.mark.parametrize("N,d,H", [(128, 64, 1), (384, 128, 2), (1152, 128, 2), (512, 128, 128)])
def test_fp8pv_tiles(fa, N, d, H):
    g = torch.Generator().manual_seed(N + 3 * d + H)
    q, k, v = (torch.randn(1, H, N, d, generator=g).to(torch.bfloat16) for _ in range(3))
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    rows = np.arange(H * N) if H * N <= 4096 else np.arange(0, H * N, 11)
    _run_fp8(fa, host64, (q.cuda(), k.cuda(), v.cuda()), rows, f"N{N} d{d} H{H}", causal=(N == 384))


@pytest.mark.parametrize("name", ["outlier_b2h16_n4096_d128", "student_t_b1h32_n8192_d128", "long_b1h32_n16384_d128"])
def test_fp8pv_full_size_sampled_rows(fa, name):
    host64, dev = load_workload(name)
    _run_fp8(fa, host64, dev, workloads.sampled_rows(name), name)


def test_fp8pv_fidelity_against_exact_attention(fa):
    """FP8 P/V is the accurate route (Table accuracy-matched-control): on the long
    workload's sampled rows its error against exact attention is well below the
    Direct-P MXFP4 route's."""
    from oracle import exact
    name = "long_b1h32_n16384_d128"
    (q, k, v), dev = load_workload(name)
    rows = workloads.sampled_rows(name)
    B, H, N, d = q.shape
    s = 1.0 / np.sqrt(d)
    ref = np.zeros((len(rows), d))
    for bh in np.unique(rows // N):
        sel = np.nonzero(rows // N == bh)[0]
        b, h = divmod(int(bh), H)
        ref[sel] = exact.attention(q[b, h][rows[sel] % N], k[b, h], v[b, h], s)
    idx = torch.from_numpy(rows).cuda()
    o4 = fa.forward_mxfp4(*gpu_operands(*dev)).reshape(-1, d)[idx].cpu().numpy()
    o8 = fa.forward_mxfp4(*fa.quantize_qkv(*dev, pv_fp8=True), pv_fp8=True).reshape(-1, d)[idx].cpu().numpy()
    m4 = exact.error_metrics(o4, ref)
    m8 = exact.error_metrics(o8, ref)
    print(f"[fidelity] MXFP4 P/V cos {m4[0]:.6f} rel-L2 {m4[1]:.6f}; FP8 P/V cos {m8[0]:.6f} rel-L2 {m8[1]:.6f}",
          flush=True)
    assert m8[0] > 0.98 and m8[1] < 0.55 * m4[1]



@pytest.mark.parametrize("where", ["q_row", "k_key", "v_column"])
def test_non_finite_input_propagation(fa, where):
    """A NaN in one input element (its 32-value block gets E8M0 byte 255, which the
    matrix unit reads as NaN) propagates as the header states, and nothing else moves:
    * Q row 5 of head 0: every score of that row is NaN, every code 0, the output row
      NaN (0/0); every other row matches the oracle.
    * K key 77 of head 1: that key's score is NaN in every row, so its code is 0 and it
      sets no block maximum: head 1 equals the oracle run with key 77 moved far below
      every other score (K row 77 = -1024 e_10 against queries whose element 10 is at
      least 1/2), which gives the key code 0 by the code map.
    * V element (77, 10) of head 1: column 10 of every row of head 1 is NaN (the V^T
      block of keys 64..95 in that column is NaN); all other columns, and head 0, match
      the oracle run with that element set to 0."""
    g = torch.Generator().manual_seed(40)
    B, H, N, d = 1, 2, 256, 64
    q, k, v = (torch.randn(B, H, N, d, generator=g) for _ in range(3))
    q[0, 1, :, 10] = q[0, 1, :, 10].abs() + 0.5
    q_ref, k_ref, v_ref = q.clone(), k.clone(), v.clone()
    nan_rows = np.zeros(B * H * N, dtype=bool)
    nan_cols = np.zeros((B * H * N, d), dtype=bool)
    if where == "q_row":
        q[0, 0, 5, 3] = float("nan")
        nan_rows[5] = True
        nan_cols[5] = True
    elif where == "k_key":
        k[0, 1, 77, 10] = float("nan")
        k_ref[0, 1, 77] = 0.0
        k_ref[0, 1, 77, 10] = -1024.0
    else:
        v[0, 1, 77, 10] = float("nan")
        v_ref[0, 1, 77, 10] = 0.0
        nan_cols[N:, 10] = True
    q, k, v, q_ref, k_ref, v_ref = (t.to(torch.bfloat16) for t in (q, k, v, q_ref, k_ref, v_ref))
    print(f"[non-finite {where}] B{B} H{H} N{N} d{d}", flush=True)
    out = fa.forward_mxfp4(*gpu_operands(q.cuda(), k.cuda(), v.cuda()))
    torch.cuda.synchronize()
    got = out.reshape(-1, d).cpu().numpy().astype(np.float64)
    print(f"[non-finite {where}] NaN entries {int(np.isnan(got).sum())}, expected {int(nan_cols.sum())}", flush=True)
    assert np.array_equal(np.isnan(got), nan_cols), "NaN entries differ from the documented propagation"
    host64 = tuple(workloads.as_f64(t) for t in (q_ref, k_ref, v_ref))
    rows = np.nonzero(~nan_rows)[0]
    ref = oracle_rows(*host64, rows, 1.0 / np.sqrt(d), want_codes=False)
    keep = ~nan_cols[rows]
    cols = np.nonzero(keep.all(axis=0))[0]          # columns finite in every checked row
    check_output(got[rows][:, cols], ref["O"][:, cols], f"non-finite {where}, finite entries")
    if where == "v_column":
        check_output(got[:N], ref["O"][:N], "non-finite v_column, head 0 all columns")


def test_one_call_attention_equals_two_steps(fa):
    """attention_mxfp4 (quantize and forward in one call) gives the same bytes as
    quantize_qkv followed by forward_mxfp4, on every route."""
    g = torch.Generator().manual_seed(31)
    q, k, v = (torch.randn(1, 2, 512, 64, generator=g).to(torch.bfloat16).cuda() for _ in range(3))
    for opts in ({}, {"causal": True}, {"ex2_pairs": 4}, {"guard": (110, 16)}, {"pv_fp8": True}):
        one = fa.attention_mxfp4(q, k, v, **opts)
        ops = fa.quantize_qkv(q, k, v, anchored="guard" in opts, pv_fp8=opts.get("pv_fp8", False))
        two = fa.forward_mxfp4(*ops, **opts)
        torch.cuda.synchronize()
        assert torch.equal(one, two), opts
