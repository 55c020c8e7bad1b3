"""CPU oracle for the Direct-P full-MXFP4 attention forward.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 NumPy
restatement of what the paper ("Hardware-Aware FP4 FlashAttention-4") says the
noncausal forward computes.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  The product path (the
HIP library under ``paper_2609_04105_amd/``) never imports, links or calls it,
and this package imports nothing from the product path.  The two share only
the seeded input generators in ``workloads/``.

Modules
-------
e2m1     E2M1 payload: magnitude table and round-to-nearest-even encoder
         (Sec. "Problem 2", E2M1 magnitude set; eq. e2m1-boundaries).
fp32     exact single-precision product / fused multiply-add on fp64 carriers
         (used where a floating-point value decides an integer code and the
         paper fixes that decision in fp32).
mxfp4    MXFP4 input quantizer: E2M1 codes + E8M0 amplitude per 32 values
         (eq. mx-scale) with the block exponent chosen by exact squared error.
directp  Direct-P attention (Sec. "Direct-P", Fix 1 and Fix 2, Alg. 2,
         eqs. ideal-code-path, affine-code-map, represented-contributions,
         represented-output), brute-force and online (tiled) forms.
guard    the sampled QK guard of Alg. 3 (Sec. "Fix 3"): anchor permutation,
         margin M, stored-scale shift L and the floored working byte.
fp8pv    MXFP4 QK with FP8 (E4M3) P and V, the paper's accuracy control and
         training route: MXFP8 quantizer, exponential P payload, represented
         denominator.
exact    textbook softmax attention (eq. attention-intro / exact-attention)
         and the online-softmax recurrence (eq. online-recurrence).
prange   the probability-format range diagnostic of Table p-range
         (NVFP4 with global factor G, and MXFP4 probabilities).

Every function is pinned by ``tests/test_oracle_*.py`` against values the
paper prints, closed forms, invariants or brute force.  ``exact.attention`` is
pinned by a scalar-loop brute force and closed forms, and
``exact.attention_online`` against it for tile widths that divide N, leave a
ragged last tile or exceed N (``tests/test_oracle_exact.py``).
"""
