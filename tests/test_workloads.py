"""The seeded input generators: determinism, shapes, dtypes, and the stated
distribution features (outlier channels, heavy tails)."""
import numpy as np
import torch

import workloads


def test_all_workloads_declared_with_paper_shapes():
    shapes = {(w.B, w.H, w.N, w.d) for w in workloads.WORKLOADS.values()}
    assert shapes == {(1, 1, 128, 64), (1, 8, 1024, 64), (2, 16, 4096, 128),
                      (1, 32, 8192, 128), (1, 32, 16384, 128)}
    assert workloads.WORKLOADS[workloads.BENCH_WORKLOAD].N == 16384


def test_generation_is_deterministic_and_typed():
    a = workloads.generate("tiny_b1h1_n128_d64")
    b = workloads.generate("tiny_b1h1_n128_d64")
    assert all(torch.equal(x, y) for x, y in zip(a, b))
    assert a[0].dtype == torch.float32 and a[0].shape == (1, 1, 128, 64)
    s = workloads.generate("small_b1h8_n1024_d64", H=2)
    assert s[0].dtype == torch.bfloat16 and s[0].shape == (1, 2, 1024, 64)
    assert not torch.equal(a[0], a[1])


def test_outlier_channels_are_shared_by_q_and_k():
    q, k, v = (workloads.as_f64(t) for t in workloads.generate("outlier_b2h16_n4096_d128", B=1, H=2, N=512))
    sq = q.reshape(-1, 128).std(axis=0)
    sk = k.reshape(-1, 128).std(axis=0)
    big_q = set(np.nonzero(sq > 4)[0])
    assert len(big_q) == 3 and big_q == set(np.nonzero(sk > 4)[0])
    assert v.std() < 1.1


def test_student_t_has_unit_variance_and_heavy_tails():
    q, _, _ = (workloads.as_f64(t) for t in workloads.generate("student_t_b1h32_n8192_d128", H=2, N=2048))
    x = q.ravel()
    assert abs(x.var() - 1.0) < 0.15
    kurt = np.mean((x - x.mean()) ** 4) / x.var() ** 2
    assert kurt > 5.0   # Gaussian: 3


def test_sampled_rows():
    r = workloads.sampled_rows("long_b1h32_n16384_d128")
    assert len(r) == 4096 and np.all(np.diff(r) > 0) and r.max() < 32 * 16384
    assert np.array_equal(r, workloads.sampled_rows("long_b1h32_n16384_d128"))
    assert len(workloads.sampled_rows("tiny_b1h1_n128_d64")) == 128


def test_random_mxfp4_operands_shapes_and_ranges():
    ops = workloads.random_mxfp4_operands(2, 3, 256, 128, seed=5)
    shapes = [(2, 3, 256, 64), (2, 3, 256, 4), (2, 3, 256, 64), (2, 3, 256, 4), (2, 3, 128, 128), (2, 3, 128, 8)]
    assert [tuple(t.shape) for t in ops] == shapes
    assert all(t.dtype == torch.uint8 for t in ops)
    for t in ops[1::2]:
        assert int(t.min()) >= 125 and int(t.max()) <= 129
    assert int(ops[0].min()) == 0 and int(ops[0].max()) == 255
    again = workloads.random_mxfp4_operands(2, 3, 256, 128, seed=5)
    assert all(torch.equal(a, b) for a, b in zip(ops, again))


def test_random_mxfp4_operand_scores_are_exact_in_fp32():
    """The oracle refuses scores that fp32 cannot hold exactly; the band's extreme
    bytes (largest magnitude codes at the largest and smallest scales) stay exact."""
    from oracle import directp, mxfp4
    ops = [t[0, 0].numpy() for t in workloads.random_mxfp4_operands(1, 1, 256, 128, seed=6)]
    directp.raw_scores(mxfp4.scaled_operand(ops[0], ops[1]), mxfp4.scaled_operand(ops[2], ops[3]))
    big = np.full((2, 64), 0x77, dtype=np.uint8)
    for sq, sk in ((129, 129), (125, 129), (125, 125)):
        q6 = mxfp4.scaled_operand(big, np.full((2, 4), sq, dtype=np.uint8))
        k6 = mxfp4.scaled_operand(big, np.full((2, 4), sk, dtype=np.uint8))
        raw = directp.raw_scores(q6, k6)
        assert np.all(raw == 128 * 36.0 * 2.0 ** (sq + sk - 254))


def test_random_mxfp8_vt_bytes_are_finite_e4m3():
    ops = workloads.random_mxfp4_operands(1, 2, 256, 64, seed=7, v_fp8=True)
    vt = ops[4]
    assert tuple(vt.shape) == (1, 2, 64, 256) and tuple(ops[5].shape) == (1, 2, 64, 8)
    assert int((vt & 0x7F).max()) == 0x7E          # 0x7f / 0xff (NaN) never drawn
    assert int((vt >> 7).min()) == 0 and int((vt >> 7).max()) == 1
    from oracle import fp8pv
    assert np.all(np.isfinite(fp8pv.dequantize(vt[0, 0].numpy(), ops[5][0, 0].numpy())))
