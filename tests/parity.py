"""Helpers shared by the GPU parity tests: oracle runs on selected rows and the
comparison metrics.  Imports the oracle (test infrastructure) and, lazily, the
HIP binding; nothing here is used by the product path."""
import numpy as np
import torch

import workloads
from oracle import directp, e2m1, mxfp4

CODE_MISMATCH_MAX = 1e-4   # fraction of Direct-P codes allowed to differ (rounding ties)
O_REL_L2_MAX = 2e-3        # output relative L2 error bound
O_COS_MIN = 0.9999         # output cosine bound
O_ROW_REL_L2_MAX = 2e-3    # the same relative L2 bound on every checked row on its own
TAU = 32                   # the forward's row reference may lag the row maximum by up to TAU binades


def oracle_rows(q, k, v, rows, softmax_scale, affine_a=1.5, affine_b=1.2, want_codes=True, ex2_pairs=0,
                causal=False, mode="affine32"):
    """Run the oracle on flattened query ``rows`` of fp64 arrays q, k, v [B, H, N, d].

    The oracle quantizes its own operands (oracle.mxfp4).  Returns a dict of
    row-aligned arrays: O, E, M, D and (optionally) codes.  ``mode`` is the
    oracle's code decision: ``affine32`` (the fp32 fused multiply-add) or
    ``affine64`` (eq. affine-code-map written out in fp64).
    """
    B, H, N, d = q.shape
    rows = np.asarray(rows, dtype=np.int64)
    heads = rows // N
    out = {"O": np.zeros((len(rows), d)), "E": np.zeros((len(rows), N // 32), dtype=np.int64),
           "M": np.zeros(len(rows), dtype=np.int64), "D": np.zeros(len(rows)), "LSE": np.zeros(len(rows))}
    if want_codes:
        out["codes"] = np.zeros((len(rows), N), dtype=np.uint8)

    def one_head(bh):
        b, h = divmod(int(bh), H)
        sel = np.nonzero(heads == bh)[0]
        local = rows[sel] % N
        qc, qs = mxfp4.quantize(q[b, h], axis=-1)
        kc, ks = mxfp4.quantize(k[b, h], axis=-1)
        vc, vs = mxfp4.quantize(v[b, h], axis=-2)
        return sel, directp.forward_rows(qc, qs, kc, ks, vc, vs, local, softmax_scale, affine_a, affine_b, mode=mode,
                                         want_codes=want_codes, ex2_pairs=ex2_pairs, causal=causal)

    for sel, res in _per_head(one_head, heads):
        for key in res:
            out[key][sel] = res[key]
    return out


def _per_head(fn, heads, workers=8):
    """fn(bh) for every head in ``heads``, on a pool of host threads (the oracle's
    NumPy work releases the interpreter lock), in head order."""
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=workers) as ex:
        return list(ex.map(fn, np.unique(heads)))


def oracle_rows_two_maps(q, k, v, rows, softmax_scale, workers=8):
    """Codes and block exponents of flattened query ``rows`` under both code
    decisions of the oracle, from one quantization of each head: ``affine64``
    (eq. affine-code-map written out in fp64, with its output O) and
    ``affine32`` (the fp32 fused multiply-add).  Heads run on a thread pool."""
    B, H, N, d = q.shape
    rows = np.asarray(rows, dtype=np.int64)
    heads = rows // N
    out = {"codes64": np.zeros((len(rows), N), dtype=np.uint8), "E64": np.zeros((len(rows), N // 32), np.int64),
           "codes32": np.zeros((len(rows), N), dtype=np.uint8), "E32": np.zeros((len(rows), N // 32), np.int64),
           "O64": np.zeros((len(rows), d))}

    def one_head(bh):
        b, h = divmod(int(bh), H)
        sel = np.nonzero(heads == bh)[0]
        local = rows[sel] % N
        qc, qs = mxfp4.quantize(q[b, h][local], axis=-1)
        kc, ks = mxfp4.quantize(k[b, h], axis=-1)
        vc, vs = mxfp4.quantize(v[b, h], axis=-2)
        res = directp.forward_rows(qc, qs, kc, ks, vc, vs, np.arange(len(local)), softmax_scale, mode="affine64")
        raw = directp.raw_scores(mxfp4.scaled_operand(qc, qs), mxfp4.scaled_operand(kc, ks))
        E32, _, k32 = directp.block_exponents_and_codes(raw, softmax_scale, 1.5, 1.2, "affine32")
        return sel, res, E32, k32

    for sel, res, E32, k32 in _per_head(one_head, heads, workers):
        out["codes64"][sel], out["E64"][sel], out["O64"][sel] = res["codes"], res["E"], res["O"]
        out["codes32"][sel], out["E32"][sel] = k32, E32
    return out


def rel_l2_cos(a, b):
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    rel = np.linalg.norm(a - b) / np.linalg.norm(b)
    cos = a @ b / (np.linalg.norm(a) * np.linalg.norm(b))
    return float(rel), float(cos)


def row_rel_l2(a, b):
    """Per-row relative L2 error ||a_i - b_i|| / ||b_i|| of [R, d] arrays.  A row
    whose reference is exactly zero counts as 0 if the row matches exactly, else inf."""
    a = np.asarray(a, dtype=np.float64).reshape(len(b), -1)
    b = np.asarray(b, dtype=np.float64).reshape(len(b), -1)
    num = np.linalg.norm(a - b, axis=1)
    den = np.linalg.norm(b, axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.where(den > 0, num / np.where(den > 0, den, 1.0), np.where(num == 0, 0.0, np.inf))


def check_output(got, ref, label):
    """The output gates: global relative L2 and cosine over all checked rows, and
    the relative L2 of every row on its own (so that an error confined to a few
    rows cannot hide in the global norm).  Returns (rel, cos, worst row rel)."""
    rel, cos = rel_l2_cos(got, ref)
    rows = row_rel_l2(got, ref)
    worst = float(rows.max()) if rows.size else 0.0
    print(f"[{label}] O rel-L2 {rel:.3e}  cos {cos:.10f}  worst row rel-L2 {worst:.3e} "
          f"(row {int(rows.argmax()) if rows.size else -1} of {len(rows)})", flush=True)
    assert rel <= O_REL_L2_MAX and cos >= O_COS_MIN, f"{label}: rel {rel} cos {cos}"
    assert worst <= O_ROW_REL_L2_MAX, f"{label}: row {int(rows.argmax())} rel-L2 {worst:.3e}"
    return rel, cos, worst


def unpack_codes(packed):
    """GPU p_codes [R, N/2] -> nibble codes [R, N] (uint8)."""
    return e2m1.unpack_nibbles(np.asarray(packed, dtype=np.uint8))


def gpu_operands(q, k, v):
    """Quantize torch GPU tensors with the HIP quantizer."""
    import paper_2609_04105_amd as fa
    return fa.quantize_qkv(q, k, v)


def load_workload(name, device="cuda", **override):
    """(q, k, v) on the CPU (workload dtype), their fp64 NumPy copies and GPU copies."""
    q, k, v = workloads.generate(name, **override)
    host64 = tuple(workloads.as_f64(t) for t in (q, k, v))
    dev = tuple(t.to(device) for t in (q, k, v))
    return host64, dev


def check_directp_dump(dump, ref, label):
    """Assert the Direct-P dump of the GPU against the oracle (codes, E, M, D)."""
    codes = unpack_codes(dump["p_codes"].cpu().numpy())
    mag = codes & 7
    neg = (codes & 8) != 0
    assert not np.any(neg & (mag != 0)), f"{label}: a nonzero P code carries a sign bit"
    mismatch = float(np.mean(mag != ref["codes"]))
    assert mismatch <= CODE_MISMATCH_MAX, f"{label}: code mismatch fraction {mismatch:.3e}"
    E = dump["block_exp"].cpu().numpy().astype(np.int64)
    seen = ref["E"] != directp.NO_BLOCK          # blocks with a visible key (causal mask)
    assert np.all(E[~seen] == -32768), f"{label}: a block without visible keys has an exponent"
    e_mismatch = float(np.mean(E[seen] != ref["E"][seen]))
    assert e_mismatch <= CODE_MISMATCH_MAX, f"{label}: block exponent mismatch fraction {e_mismatch:.3e}"
    M = dump["row_m"].cpu().numpy().astype(np.int64)
    assert np.all((M <= ref["M"]) & (M >= ref["M"] - TAU)), f"{label}: row reference outside [M - {TAU}, M]"
    D = dump["row_d"].cpu().numpy().astype(np.float64) * np.exp2(M - ref["M"])
    rel = np.abs(D - ref["D"]) / ref["D"]
    assert rel.max() < 1e-4, f"{label}: denominator rel error {rel.max():.3e}"
    return mismatch


def oracle_rows_guarded(q, k, v, rows, softmax_scale, margin, shift, ex2_pairs=0):
    """The guarded oracle (Alg. 3) on flattened query ``rows`` of fp64 q, k, v
    [B, H, N, d] in their ORIGINAL key order: K and V are put in anchor order
    here, as the anchored quantizer does on the GPU."""
    from oracle import guard
    B, H, N, d = q.shape
    perm = guard.anchor_permutation(N)
    rows = np.asarray(rows, dtype=np.int64)
    heads = rows // N
    out = {"O": np.zeros((len(rows), d)), "ebar": np.zeros((len(rows), N // 32), dtype=np.int64),
           "D": np.zeros(len(rows)), "LSE": np.zeros(len(rows)), "codes": np.zeros((len(rows), N), dtype=np.uint8)}
    def one_head(bh):
        b, h = divmod(int(bh), H)
        sel = np.nonzero(heads == bh)[0]
        local = rows[sel] % N
        qc, qs = mxfp4.quantize(q[b, h][local], axis=-1)
        kc, ks = mxfp4.quantize(k[b, h][perm], axis=-1)
        vc, vs = mxfp4.quantize(v[b, h][perm], axis=-2)
        return sel, guard.forward_rows(qc, qs, kc, ks, vc, vs, np.arange(len(local)), softmax_scale, margin, shift,
                                       ex2_pairs=ex2_pairs)

    for sel, res in _per_head(one_head, heads):
        for key in out:
            out[key][sel] = res[key]
    return out


def check_guarded_dump(dump, ref, label):
    """Assert the guarded Direct-P dump against the oracle: codes, working exponents
    (decided in the same fp32 steps, so exact), and the denominator."""
    codes = unpack_codes(dump["p_codes"].cpu().numpy())
    mag = codes & 7
    assert not np.any(((codes & 8) != 0) & (mag != 0)), f"{label}: a nonzero P code carries a sign bit"
    mismatch = float(np.mean(mag != ref["codes"]))
    assert mismatch <= CODE_MISMATCH_MAX, f"{label}: code mismatch fraction {mismatch:.3e}"
    E = dump["block_exp"].cpu().numpy().astype(np.int64)
    assert np.array_equal(E, ref["ebar"]), f"{label}: working exponents differ"
    assert np.all(dump["row_m"].cpu().numpy() == 0)
    D = dump["row_d"].cpu().numpy().astype(np.float64)
    rel = np.abs(D - ref["D"]) / ref["D"]
    assert rel.max() < 1e-4, f"{label}: denominator rel error {rel.max():.3e}"
    return mismatch


def oracle_rows_fp8(q, k, v, rows, softmax_scale, causal=False):
    """The FP8-P/V oracle (MXFP4 QK, E4M3 P, MXFP8 V) on flattened query ``rows``."""
    from oracle import fp8pv
    B, H, N, d = q.shape
    rows = np.asarray(rows, dtype=np.int64)
    heads = rows // N
    out = {"O": np.zeros((len(rows), d)), "E": np.zeros((len(rows), N // 32), dtype=np.int64),
           "M": np.zeros(len(rows), dtype=np.int64), "D": np.zeros(len(rows)), "LSE": np.zeros(len(rows)),
           "codes": np.zeros((len(rows), N), dtype=np.uint8)}
    def one_head(bh):
        b, h = divmod(int(bh), H)
        sel = np.nonzero(heads == bh)[0]
        qc, qs = mxfp4.quantize(q[b, h], axis=-1)
        kc, ks = mxfp4.quantize(k[b, h], axis=-1)
        vc, vs = fp8pv.quantize(v[b, h], axis=-2)
        return sel, fp8pv.forward_rows(qc, qs, kc, ks, vc, vs, rows[sel] % N, softmax_scale, causal=causal)

    for sel, res in _per_head(one_head, heads):
        for key in out:
            out[key][sel] = res[key]
    return out


def check_fp8_dump(dump, ref, label):
    """FP8 route: E4M3 payload bytes (non-negative), block exponents, row reference
    within the lazy window, and the denominator."""
    codes = dump["p_codes"].cpu().numpy()
    assert not np.any(codes & 0x80), f"{label}: a P payload carries a sign bit"
    mismatch = float(np.mean(codes != ref["codes"]))
    assert mismatch <= CODE_MISMATCH_MAX, f"{label}: payload mismatch fraction {mismatch:.3e}"
    E = dump["block_exp"].cpu().numpy().astype(np.int64)
    seen = ref["E"] != directp.NO_BLOCK
    assert np.all(E[~seen] == -32768)
    assert float(np.mean(E[seen] != ref["E"][seen])) <= CODE_MISMATCH_MAX
    M = dump["row_m"].cpu().numpy().astype(np.int64)
    assert np.all((M <= ref["M"]) & (M >= ref["M"] - TAU)), f"{label}: row reference outside [M - {TAU}, M]"
    D = dump["row_d"].cpu().numpy().astype(np.float64) * np.exp2(M - ref["M"])
    rel = np.abs(D - ref["D"]) / ref["D"]
    # E4M3 payload sums are not exact in fp32 (E2M1 code sums are): the bound of
    # recursive fp32 summation of N positive terms, N * 2^-24
    tol = max(1e-4, codes.shape[1] * 2.0 ** -24)
    assert rel.max() < tol, f"{label}: denominator rel error {rel.max():.3e} (bound {tol:.1e})"
    return mismatch
