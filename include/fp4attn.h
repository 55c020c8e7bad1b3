/*
 * fp4attn: noncausal full-MXFP4 attention forward with Direct-P probabilities
 * on AMD Instinct MI355X (gfx950).
 *
 * Method: "Hardware-Aware FP4 FlashAttention-4" (arXiv 2609.04105).  The
 * forward computes S = Q K^T / sqrt(d), P = softmax(S), O = P V
 * (eq. attention-intro) with Q, K, P and V all in MXFP4: E2M1 codes plus one
 * E8M0 amplitude per 32 values (Sec. "Problem 2", Table fp4-formats,
 * eq. mx-scale).  P is produced by Direct-P (Sec. "Direct-P", Alg. 2): scores
 * map straight to E2M1 codes through an affine classifier (eq. affine-code-map)
 * and the row normaliser is the sum of the same rounded codes that the PV
 * product consumes (Fix 2, eqs. represented-contributions/-output).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensor pointers are DEVICE pointers owned by the caller; the library never
 *   allocates, frees or keeps them.  Every pointer must be 16-byte aligned.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream of
 *   the current device).  The work runs on the device that `stream` belongs
 *   to, and every pointer must be memory of that device (or mapped into it).
 *   Arguments are validated synchronously on the host; on success the work is
 *   enqueued asynchronously on `stream` and the call returns without waiting.
 *   On any error nothing is enqueued and the outputs are untouched.
 * - Outputs are fully overwritten; inputs are never written.
 * - The library holds no global state besides a thread-local error string and
 *   is safe to call from several host threads.
 * - MXFP4 layout: E2M1 code = sign << 3 | k, k indexing {0, .5, 1, 1.5, 2, 3,
 *   4, 6}; two codes per byte, element 2j in bits 3:0 and element 2j+1 in bits
 *   7:4.  E8M0 byte u: amplitude 2^(u-127), u = 255 is NaN.  A value is
 *   represented as 2^(u-127) * e2m1(code) / 6: the byte stores the block
 *   amplitude, not the step (eq. mx-scale).
 */
#ifndef FP4ATTN_H
#define FP4ATTN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FP4ATTN_OK = 0,
  FP4ATTN_ERR_INVALID_ARG = 1, /* null/misaligned pointer, bad size, enum or scalar */
  FP4ATTN_ERR_UNSUPPORTED = 2, /* valid but not implemented (head dim not 64 or 128, N above 2^22, ...) */
  FP4ATTN_ERR_HIP = 3          /* the HIP runtime refused the launch; see fp4attn_last_error() */
} fp4attn_status;

typedef enum {
  FP4ATTN_F32 = 0,
  FP4ATTN_BF16 = 1
} fp4attn_dtype;

/*
 * MXFP4 quantizer (eq. mx-scale).  Quantizes `batch` row-major [rows, cols]
 * matrices of `src_dtype` in blocks of 32 consecutive values along `axis`.
 *
 *   axis = 1 (Q, K: [N, d]):  codes [batch, rows, cols/2], scales [batch, rows, cols/32].
 *   axis = 0 (V: [N, d], blocks along the sequence): stored TRANSPOSED,
 *            codes [batch, cols, rows/2], scales [batch, cols, rows/32].
 *
 * Per block with absolute maximum a > 0 the amplitude is 2^floor(log2 a) or
 * 2^ceil(log2 a) (the two candidates of eq. mx-scale), whichever gives the
 * smaller squared reconstruction error over the block (ties: the ceiling),
 * compared exactly.  Exponents clamp to [-127, 127].  An all-zero block gets
 * u = 0; a block holding NaN or +-Inf gets u = 255 and zero codes.  The sign bit
 * of each code is the sign bit of its input (so -0.0 encodes as 0x8).
 *
 * Errors: INVALID_ARG if a pointer is null or misaligned, batch < 1, rows < 1,
 * cols < 1, the blocked extent (cols for axis 1, rows for axis 0) is not a
 * multiple of 32, axis is not 0 or 1, src_dtype is not a fp4attn_dtype, or
 * the tensor holds more than 2^40 blocks of 32.
 * The quantizer is not part of the timed forward (the paper times the kernel
 * on prequantized operands).
 */
fp4attn_status fp4attn_quantize_mxfp4(const void* src, int src_dtype, int64_t batch, int64_t rows,
                                      int64_t cols, int axis, uint8_t* codes, uint8_t* scales,
                                      void* stream);

/*
 * MXFP8 quantizer for the FP8 P/V route: E4M3 payload (bias 7, three mantissa
 * bits, largest finite 448, subnormals kept) plus one E8M0 byte per 32 values
 * along `axis`, with the layouts of fp4attn_quantize_mxfp4 but one code byte
 * per value:
 *
 *   axis = 1: codes [batch, rows, cols],  scales [batch, rows, cols/32].
 *   axis = 0: codes [batch, cols, rows] (transposed), scales [batch, cols, rows/32].
 *
 * The amplitude of a block is the smallest power of two 2^e with
 * max|v| / 2^e <= 448 (no payload saturates); codes are v / 2^e rounded to the
 * nearest E4M3 value, ties to even, sign bit 7 = the input's sign bit.  Zero
 * block: u = 0; non-finite block: u = 255, zero codes.  The represented value
 * is 2^(u-127) * e4m3(code).  Errors: as fp4attn_quantize_mxfp4.
 */
fp4attn_status fp4attn_quantize_mxfp8(const void* src, int src_dtype, int64_t batch, int64_t rows,
                                      int64_t cols, int axis, uint8_t* codes, uint8_t* scales,
                                      void* stream);

/*
 * fp4attn_quantize_mxfp4 of the rows put in anchor order first (Sec. "Fix 3":
 * before the launch, globally distributed K/V rows move into the first key
 * tile; exact attention does not change).  Row r of the quantized matrix is
 * source row pi(r): for r < n_anchor, r * (rows / n_anchor) (evenly spread
 * anchors); the remaining rows follow in their original order.  Used for K
 * (axis 1) and V (axis 0, so V's 32-key blocks follow the new key order) of
 * the guarded forward, with n_anchor = 128 (its first key tile).
 *
 * Errors: those of fp4attn_quantize_mxfp4, plus INVALID_ARG if n_anchor < 1 or
 * n_anchor does not divide rows.
 */
fp4attn_status fp4attn_quantize_mxfp4_anchored(const void* src, int src_dtype, int64_t batch,
                                               int64_t rows, int64_t cols, int axis, int64_t n_anchor,
                                               uint8_t* codes, uint8_t* scales, void* stream);

/*
 * Direct-P full-MXFP4 attention forward, noncausal (Sec. "Direct-P", Alg. 2,
 * eqs. affine-code-map, represented-contributions, represented-output).
 *
 *   q_codes  [B, H, N, d/2]  q_scales  [B, H, N, d/32]   (fp4attn_quantize_mxfp4, axis 1)
 *   k_codes  [B, H, N, d/2]  k_scales  [B, H, N, d/32]   (axis 1)
 *   vt_codes [B, H, d, N/2]  vt_scales [B, H, d, N/32]   (V quantized with axis 0)
 *   out      [B, H, N, d] of out_dtype (FP4ATTN_F32 or FP4ATTN_BF16)
 *
 * For query row i and 32-key block B the kernel forms the score
 * y = raw * softmax_scale * log2(e) / 36 (raw = the block-scaled FP4 product,
 * 36 Qhat.Khat), the block exponent E_B = floor(max_B y), and the codes
 * q = E2M1(max(0, A (y - E_B + log2 6) + B)) with A = affine_a, B = affine_b
 * (the paper's `fast` fit is 1.5 / 1.2), evaluated as one fp32 fused
 * multiply-add per score.  P enters the PV product as MXFP4 with E8M0 byte
 * E_B - M_i + 127 against an integer running row reference M_i (clamped to
 * [0, 254]; 0 marks a block more than 127 binades below the reference), and
 * O_i = sum_B 2^(E_B - M_i) sum_j q_ij Vhat_j / sum_B 2^(E_B - M_i) c_B with
 * c_B = sum_j q_ij taken from the same codes.
 *
 * Errors: INVALID_ARG for null/misaligned pointers, B < 1, H < 1, N < 128 or
 * N % 128 != 0, softmax_scale not finite or <= 0, affine_a not finite or <= 0,
 * affine_b not finite, bad out_dtype, B*H*N beyond 2^31 - 1 or B*H beyond
 * 16776960 (65535 * 256).  UNSUPPORTED for
 * d not in {64, 128} or N above 4194304 (2^22) keys.
 *
 * Non-finite inputs (a block whose E8M0 byte is 255, as the quantizers write for a
 * block holding NaN or +-Inf; the matrix unit reads that byte as NaN) never fault
 * and stay within their head: a non-finite Q block makes every score of its row
 * NaN, every code of the row 0 and the output row NaN (0/0); a non-finite K block
 * makes its key's score NaN in every row, which the code map sends to code 0 and
 * the block maximum skips, so each row is the forward over the other keys; a
 * non-finite V^T block (32 keys of one column) makes that column NaN in every row
 * of the head.  The extended routes promise only that they do not fault.
 */
fp4attn_status fp4attn_forward_mxfp4(const uint8_t* q_codes, const uint8_t* q_scales,
                                     const uint8_t* k_codes, const uint8_t* k_scales,
                                     const uint8_t* vt_codes, const uint8_t* vt_scales,
                                     int64_t B, int64_t H, int64_t N, int64_t d,
                                     float softmax_scale, float affine_a, float affine_b,
                                     void* out, int out_dtype, void* stream);

/*
 * Options of the extended forward.  Fill with fp4attn_forward_options_init()
 * and then change fields; struct_size must equal sizeof(fp4attn_forward_options)
 * of the header the caller was built with.
 *
 *   affine_a, affine_b  the affine code map (init 1.5 / 1.2, the `fast` fit).
 *   ex2_pairs           native-exponential mixing (Sec. "Fix 1": a selected
 *                       pair may take the native exponential; Table
 *                       policy-definition: the `accurate` policy does so on
 *                       about a quarter of pair positions).  k in {0, 1, 2, 4,
 *                       8, 16} of the 16 key pairs of every 32-key block (pair
 *                       p = keys 2p, 2p+1, selected iff p % (16 / k) == 0) get
 *                       the ideal code q = E2M1(2^x), x = y - E_B + log2 6
 *                       evaluated as one fp32 fma, 2^x on the hardware
 *                       exponential; the other pairs keep the affine map.
 *                       init 0 (all affine); 16 is the exp2-only route.
 *   guard               1: the sampled QK guard of Alg. 3 replaces the online
 *                       row reference.  The first 128 keys are the anchor set
 *                       (K and V quantized with
 *                       fp4attn_quantize_mxfp4_anchored, n_anchor = 128); per
 *                       row, with y = raw * softmax_scale * log2(e) / 36 in
 *                       fp32 and Y = the largest y over the anchors, the
 *                       reference is R = fp32(Y + guard_margin), the block
 *                       exponent e_B = floor(fp32(max_B y - R)), the working
 *                       byte ubar_B = clamp(e_B + 127, guard_shift + 1, 254)
 *                       (floored before the codes are formed), the codes
 *                       those of Alg. 2 with x = y - T + log2 6,
 *                       T = fp32(R + ubar_B - 127), and the published E8M0
 *                       byte ubar_B - guard_shift.  init 0.  Built for
 *                       ex2_pairs 0, 4 and 16.
 *   guard_margin        M, guard_shift  L: integers >= 0 with M + L <= 126
 *                       (Alg. 3 step 2); init 110 / 16, the paper's setting
 *                       for its 1.3B video model.
 *   causal              1: query i sees keys j <= i only (the forward of the
 *                       paper's causal-training route, Sec. "Pass the forward
 *                       quantization into backward"); hidden scores take code
 *                       0.  init 0.  Built for ex2_pairs 0, 4 and 16; not with
 *                       the guard.
 *   pv_fp8              1: P and V are FP8 (E4M3) instead of E2M1 (the
 *                       paper's FP8 probability/value route, its accuracy
 *                       control and training choice).  vt_codes/vt_scales then
 *                       come from fp4attn_quantize_mxfp8 with axis 0 (codes
 *                       [B, H, d, N], one byte per value).  P payload of key j
 *                       in block B: E4M3(2^(y_j - E_B + 7)), exponential on
 *                       every key, block maximum in [128, 256); E8M0 byte
 *                       E_B - M_i + 120; the denominator sums the same
 *                       payloads.  init 0.  Not with the guard or ex2_pairs.
 *   lse                 optional DEVICE pointer (NULL: not written) to
 *                       [B, H, N] fp32: the natural-log row normaliser the
 *                       backward reconstructs probabilities from, for the
 *                       represented operator: LSE_i = ref_i ln 2 + ln(D_i / 6)
 *                       where D_i is the represented denominator relative to
 *                       2^ref_i, ref_i = M_i (online reference) or R_i + L
 *                       (guard); exp(z_ij - LSE_i) is then the represented
 *                       probability of key j.  (FP8 route: LSE_i = M_i ln 2 +
 *                       ln D_i, D_i carrying the payload's 2^-7.)  init NULL.
 */
typedef struct fp4attn_forward_options {
  uint32_t struct_size;
  float affine_a;
  float affine_b;
  int32_t ex2_pairs;
  int32_t guard;
  int32_t guard_margin;
  int32_t guard_shift;
  int32_t causal;
  int32_t pv_fp8;
  float* lse;
} fp4attn_forward_options;

/* Writes the defaults listed above (and struct_size) into *opts; NULL is ignored. */
void fp4attn_forward_options_init(fp4attn_forward_options* opts);

/*
 * fp4attn_forward_mxfp4 with options (NULL = the defaults).  Operands, layout
 * and output as fp4attn_forward_mxfp4.  Errors: those of fp4attn_forward_mxfp4,
 * plus INVALID_ARG for a struct_size other than sizeof(fp4attn_forward_options),
 * ex2_pairs outside {0, 1, 2, 4, 8, 16}, guard or causal not 0 or 1, a guard
 * margin and shift outside the budget, or an lse pointer that is not 16-byte
 * aligned; UNSUPPORTED for the guard or the causal mask with ex2_pairs not in
 * {0, 4, 16}, or both together, and for pv_fp8 with the guard or ex2_pairs.
 */
fp4attn_status fp4attn_forward_mxfp4_ex(const uint8_t* q_codes, const uint8_t* q_scales,
                                        const uint8_t* k_codes, const uint8_t* k_scales,
                                        const uint8_t* vt_codes, const uint8_t* vt_scales,
                                        int64_t B, int64_t H, int64_t N, int64_t d,
                                        float softmax_scale, const fp4attn_forward_options* opts,
                                        void* out, int out_dtype, void* stream);

/*
 * Same-design BF16 attention forward: the speed baseline of the paper's
 * canonical speedup t_BF16 / t_k (eq. canonical-speedup).  Textbook softmax
 * attention (eq. exact-attention) with the online recurrence
 * (eq. online-recurrence) in base 2, fp32 accumulation, P rounded to bf16 for
 * the PV product, and the row sum taken over those same rounded values.
 *
 *   q, k, v [B, H, N, d] bf16 (row-major, the same layout for all three);
 *   out [B, H, N, d] of out_dtype.
 *
 * Errors: as fp4attn_forward_mxfp4 (no affine arguments).
 */
fp4attn_status fp4attn_forward_bf16(const void* q, const void* k, const void* v,
                                    int64_t B, int64_t H, int64_t N, int64_t d,
                                    float softmax_scale, void* out, int out_dtype, void* stream);

/*
 * Test hook: runs exactly the forward kernel of fp4attn_forward_mxfp4_ex (same
 * launch configuration and arguments, `opts` NULL = the defaults, writes `out`
 * too) and additionally
 * dumps the Direct-P state of selected query rows (Alg. 2, steps 1-6):
 *
 *   row_ids    [n_rows] int64, flattened (b*H + h)*N + i, STRICTLY ASCENDING
 *              (rows not found by the kernel's binary search are not dumped)
 *   p_codes    [n_rows, N/2]  the P codes fed to the PV product, nibble-packed
 *              ([n_rows, N] E4M3 bytes with pv_fp8)
 *   block_exp  [n_rows, N/32] int16 absolute block exponents E_B (-32768:
 *              the block has no visible key under the causal mask)
 *   row_m      [n_rows] int32 final integer row reference M_i (0 under the guard);
 *              it lags the row's largest block exponent by at most 32 binades
 *   row_d      [n_rows] fp32 represented denominator relative to 2^M_i (under
 *              the guard: sum_B 2^(u'_B - 127) c_B with the published bytes)
 *              (block_exp holds the working exponents ubar_B - 127 under the guard)
 *   wg_clock   optional (NULL: not written), [B*H*N/128][2] uint64: workgroup
 *              w of the launch writes entry [w][0], the shader-clock cycles
 *              it was resident, and [w][1], the same interval in ticks of the
 *              100 MHz constant clock; entries past the launch's workgroup
 *              count (B*H*N/256 workgroups when 256-row tiles are used) are
 *              left untouched.  Their ratio is the achieved shader clock.
 *
 * With n_rows = 0 nothing is dumped (the five dump pointers are ignored and
 * may be NULL) and the launch is the plain forward kernel itself, so wg_clock
 * then records the clock of exactly the timed kernel.
 *
 * Errors: as fp4attn_forward_mxfp4_ex, plus INVALID_ARG for n_rows < 0, a null
 * dump pointer when n_rows > 0, or a wg_clock that is not 16-byte aligned.
 */
fp4attn_status fp4attn_debug_directp_mxfp4(const uint8_t* q_codes, const uint8_t* q_scales,
                                           const uint8_t* k_codes, const uint8_t* k_scales,
                                           const uint8_t* vt_codes, const uint8_t* vt_scales,
                                           int64_t B, int64_t H, int64_t N, int64_t d,
                                           float softmax_scale, const fp4attn_forward_options* opts,
                                           void* out, int out_dtype,
                                           const int64_t* row_ids, int64_t n_rows,
                                           uint8_t* p_codes, int16_t* block_exp,
                                           int32_t* row_m, float* row_d, uint64_t* wg_clock,
                                           void* stream);

/*
 * Measurement hook: the sustained rate of the scaled FP4 matrix unit on given
 * operands, the ceiling the forward's two products are compared against.
 * Launches `blocks` x 256 threads; thread t keeps the four 16-byte fragments
 * a_codes[64 t, 64 t + 64) and the four b_codes[64 t, 64 t + 64) (E2M1 codes,
 * two per byte) in registers, issues `iters` rounds of four independent
 * 32x32x64 FP4 products with E8M0 scale bytes 127 (fragment i of A with
 * fragment (i + 1) % 4 of B), and writes the sum of its sixteen-element
 * accumulators to out[t].  Work: blocks * 256 / 64 waves * iters * 4 products
 * of 2 * 32 * 32 * 64 flop.  a_codes and b_codes hold blocks * 256 * 64
 * bytes each, out blocks * 256 floats.  Errors: INVALID_ARG for null or
 * misaligned pointers, blocks outside [1, 65535], iters < 1.
 */
fp4attn_status fp4attn_debug_mfma_stream(const uint8_t* a_codes, const uint8_t* b_codes, int blocks, int iters,
                                         float* out, void* stream);

/* Static description of a status code; never NULL. */
const char* fp4attn_status_string(int status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* fp4attn_last_error(void);

/* ABI version of this header, (major << 16) | minor: 2.0 (fp4attn_forward_bf16
 * takes V as [B, H, N, d]; 1.x took V transposed). */
int fp4attn_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FP4ATTN_H */
