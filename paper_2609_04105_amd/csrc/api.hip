// C-ABI of libfp4attn: argument validation, status codes, and launch.
// Declarations and the contract of every entry point are in include/fp4attn.h.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "../../include/fp4attn.h"
#include "launch.hpp"

namespace {

thread_local char g_last_error[512] = "";

fp4attn_status fail(fp4attn_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
fp4attn_status fail(fp4attn_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

fp4attn_status ok() {
  g_last_error[0] = '\0';
  return FP4ATTN_OK;
}

fp4attn_status from_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(FP4ATTN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE_PTR(p)                                                                        \
  do {                                                                                        \
    if (!aligned16(p)) return fail(FP4ATTN_ERR_INVALID_ARG, "%s is null or not 16-byte aligned", #p); \
  } while (0)

constexpr int64_t kMaxN = int64_t(1) << 22;

// Shared checks of the two attention forwards.
fp4attn_status check_attention_shape(int64_t B, int64_t H, int64_t N, int64_t d, float softmax_scale, int out_dtype) {
  if (B < 1 || H < 1) return fail(FP4ATTN_ERR_INVALID_ARG, "B=%lld and H=%lld must be >= 1", (long long)B, (long long)H);
  if (N < 128 || N % 128 != 0)
    return fail(FP4ATTN_ERR_INVALID_ARG, "N=%lld must be a positive multiple of 128", (long long)N);
  if (!std::isfinite(softmax_scale) || softmax_scale <= 0.0f)
    return fail(FP4ATTN_ERR_INVALID_ARG, "softmax_scale must be finite and positive");
  if (out_dtype != FP4ATTN_F32 && out_dtype != FP4ATTN_BF16)
    return fail(FP4ATTN_ERR_INVALID_ARG, "out_dtype %d is not FP4ATTN_F32 or FP4ATTN_BF16", out_dtype);
  // B and H first, so that no product below can overflow 64 bits
  if (B > 65535 * 256 || H > 65535 * 256 || B * H > 65535 * 256 || B * H > ((int64_t(1) << 31) - 1) / N)
    return fail(FP4ATTN_ERR_INVALID_ARG, "B=%lld H=%lld N=%lld: B*H*N must stay below 2^31 and B*H below 2^24",
                (long long)B, (long long)H, (long long)N);
  if (d != 64 && d != 128) return fail(FP4ATTN_ERR_UNSUPPORTED, "head dimension d=%lld is not 64 or 128", (long long)d);
  // one head's operands (FP8 V^T: d N bytes) and every in-head byte offset stay below 2^31
  if (N > kMaxN) return fail(FP4ATTN_ERR_UNSUPPORTED, "N=%lld exceeds %lld keys", (long long)N, (long long)kMaxN);
  return FP4ATTN_OK;
}

fp4attn_status check_directp(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                             const uint8_t* k_scales, const uint8_t* vt_codes, const uint8_t* vt_scales, int64_t B,
                             int64_t H, int64_t N, int64_t d, float softmax_scale, float affine_a, float affine_b,
                             void* out, int out_dtype) {
  REQUIRE_PTR(q_codes);
  REQUIRE_PTR(q_scales);
  REQUIRE_PTR(k_codes);
  REQUIRE_PTR(k_scales);
  REQUIRE_PTR(vt_codes);
  REQUIRE_PTR(vt_scales);
  REQUIRE_PTR(out);
  if (!std::isfinite(affine_a) || affine_a <= 0.0f)
    return fail(FP4ATTN_ERR_INVALID_ARG, "affine_a must be finite and positive");
  if (!std::isfinite(affine_b)) return fail(FP4ATTN_ERR_INVALID_ARG, "affine_b must be finite");
  return check_attention_shape(B, H, N, d, softmax_scale, out_dtype);
}

fp4attn_forward_options default_options() {
  fp4attn_forward_options o{};
  o.struct_size = sizeof(fp4attn_forward_options);
  o.affine_a = 1.5f;
  o.affine_b = 1.2f;
  o.ex2_pairs = 0;
  o.guard = 0;
  o.guard_margin = 110;
  o.guard_shift = 16;
  o.causal = 0;
  o.pv_fp8 = 0;
  o.lse = nullptr;
  return o;
}

// Options of the extended entry points: NULL means the defaults.
fp4attn_status check_options(const fp4attn_forward_options* opts, fp4attn_forward_options* out) {
  if (opts == nullptr) {
    *out = default_options();
    return FP4ATTN_OK;
  }
  if (opts->struct_size != sizeof(fp4attn_forward_options))
    return fail(FP4ATTN_ERR_INVALID_ARG, "options struct_size %u, expected %zu", opts->struct_size,
                sizeof(fp4attn_forward_options));
  const int k = opts->ex2_pairs;
  if (k != 0 && k != 1 && k != 2 && k != 4 && k != 8 && k != 16)
    return fail(FP4ATTN_ERR_INVALID_ARG, "ex2_pairs=%d is not one of 0, 1, 2, 4, 8, 16", k);
  if (opts->guard != 0 && opts->guard != 1) return fail(FP4ATTN_ERR_INVALID_ARG, "guard must be 0 or 1");
  if (opts->guard) {
    if (opts->guard_margin < 0 || opts->guard_shift < 0 || opts->guard_margin + opts->guard_shift > 126)
      return fail(FP4ATTN_ERR_INVALID_ARG, "guard margin %d and shift %d must be >= 0 with margin + shift <= 126",
                  opts->guard_margin, opts->guard_shift);
    if (k != 0 && k != 4 && k != 16)
      return fail(FP4ATTN_ERR_UNSUPPORTED, "the guarded forward is built for ex2_pairs 0, 4 and 16, not %d", k);
  }
  if (opts->causal != 0 && opts->causal != 1) return fail(FP4ATTN_ERR_INVALID_ARG, "causal must be 0 or 1");
  if (opts->causal) {
    if (opts->guard) return fail(FP4ATTN_ERR_UNSUPPORTED, "the causal forward has no sampled guard");
    if (k != 0 && k != 4 && k != 16)
      return fail(FP4ATTN_ERR_UNSUPPORTED, "the causal forward is built for ex2_pairs 0, 4 and 16, not %d", k);
  }
  if (opts->pv_fp8 != 0 && opts->pv_fp8 != 1) return fail(FP4ATTN_ERR_INVALID_ARG, "pv_fp8 must be 0 or 1");
  if (opts->pv_fp8 && (opts->guard || k != 0))
    return fail(FP4ATTN_ERR_UNSUPPORTED, "the FP8 P/V route takes neither the guard nor ex2_pairs");
  if (opts->lse != nullptr && !aligned16(opts->lse))
    return fail(FP4ATTN_ERR_INVALID_ARG, "lse is not 16-byte aligned");
  *out = *opts;
  return FP4ATTN_OK;
}

void set_options(fp4attn::DirectPArgs& a, const fp4attn_forward_options& o) {
  a.ex2_pairs = o.ex2_pairs;
  a.guard = o.guard;
  a.guard_margin = o.guard_margin;
  a.guard_shift = o.guard_shift;
  a.causal = o.causal;
  a.pv_fp8 = o.pv_fp8;
  a.lse = o.lse;
}

fp4attn::DirectPArgs directp_args(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                                  const uint8_t* k_scales, const uint8_t* vt_codes, const uint8_t* vt_scales,
                                  int64_t B, int64_t H, int64_t N, int64_t d, float softmax_scale, float affine_a,
                                  float affine_b, void* out, int out_dtype) {
  fp4attn::DirectPArgs a{};
  a.q_codes = q_codes;
  a.q_scales = q_scales;
  a.k_codes = k_codes;
  a.k_scales = k_scales;
  a.vt_codes = vt_codes;
  a.vt_scales = vt_scales;
  a.out = out;
  a.B = (int)B;
  a.H = (int)H;
  a.N = (int)N;
  a.d = (int)d;
  a.out_bf16 = out_dtype == FP4ATTN_BF16;
  a.softmax_scale = softmax_scale;
  a.affine_a = affine_a;
  a.affine_b = affine_b;
  return a;
}

fp4attn_status quantize_common(const void* src, int src_dtype, int64_t batch, int64_t rows, int64_t cols, int axis,
                               int64_t n_anchor, uint8_t* codes, uint8_t* scales, void* stream, bool fp8 = false) {
  REQUIRE_PTR(src);
  REQUIRE_PTR(codes);
  REQUIRE_PTR(scales);
  if (src_dtype != FP4ATTN_F32 && src_dtype != FP4ATTN_BF16)
    return fail(FP4ATTN_ERR_INVALID_ARG, "src_dtype %d is not FP4ATTN_F32 or FP4ATTN_BF16", src_dtype);
  if (axis != 0 && axis != 1) return fail(FP4ATTN_ERR_INVALID_ARG, "axis %d must be 0 or 1", axis);
  if (batch < 1 || rows < 1 || cols < 1) return fail(FP4ATTN_ERR_INVALID_ARG, "batch, rows and cols must be >= 1");
  const int64_t blocked = axis == 1 ? cols : rows, other = axis == 1 ? rows : cols;
  if (blocked % 32 != 0)
    return fail(FP4ATTN_ERR_INVALID_ARG, "the blocked extent (%lld) must be a multiple of 32", (long long)blocked);
  // divisions instead of products, so that no check can overflow 64 bits
  const int64_t kMaxBlocks = int64_t(1) << 40;
  if (other > kMaxBlocks / batch || blocked / 32 > kMaxBlocks / (batch * other))
    return fail(FP4ATTN_ERR_INVALID_ARG, "tensor too large");
  if ((batch * other * (blocked / 32) + 255) / 256 > 0x7fffffff)
    return fail(FP4ATTN_ERR_INVALID_ARG, "tensor too large for one launch");
  if (fp8)
    return from_hip(fp4attn::launch_quantize_mxfp8(src, src_dtype, batch, rows, cols, axis, codes, scales,
                                                   static_cast<hipStream_t>(stream)),
                    "quantize launch");
  return from_hip(fp4attn::launch_quantize_mxfp4(src, src_dtype, batch, rows, cols, axis, n_anchor, codes, scales,
                                                 static_cast<hipStream_t>(stream)),
                  "quantize launch");
}

}  // namespace

namespace fp4attn {
// mfma_stream.hip: blocks x 256 threads; a and b hold 64 bytes per thread, out one float per thread.
hipError_t launch_mfma_stream(const void* a, const void* b, int blocks, int iters, float* out, hipStream_t stream);
}  // namespace fp4attn

extern "C" {

fp4attn_status fp4attn_quantize_mxfp4(const void* src, int src_dtype, int64_t batch, int64_t rows, int64_t cols,
                                      int axis, uint8_t* codes, uint8_t* scales, void* stream) {
  return quantize_common(src, src_dtype, batch, rows, cols, axis, 0, codes, scales, stream);
}

fp4attn_status fp4attn_quantize_mxfp8(const void* src, int src_dtype, int64_t batch, int64_t rows, int64_t cols,
                                      int axis, uint8_t* codes, uint8_t* scales, void* stream) {
  return quantize_common(src, src_dtype, batch, rows, cols, axis, 0, codes, scales, stream, true);
}

fp4attn_status fp4attn_quantize_mxfp4_anchored(const void* src, int src_dtype, int64_t batch, int64_t rows,
                                               int64_t cols, int axis, int64_t n_anchor, uint8_t* codes,
                                               uint8_t* scales, void* stream) {
  if (n_anchor < 1 || rows % n_anchor != 0)
    return fail(FP4ATTN_ERR_INVALID_ARG, "n_anchor=%lld must be >= 1 and divide rows=%lld", (long long)n_anchor,
                (long long)rows);
  return quantize_common(src, src_dtype, batch, rows, cols, axis, n_anchor, codes, scales, stream);
}

fp4attn_status fp4attn_forward_mxfp4(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                                     const uint8_t* k_scales, const uint8_t* vt_codes, const uint8_t* vt_scales,
                                     int64_t B, int64_t H, int64_t N, int64_t d, float softmax_scale, float affine_a,
                                     float affine_b, void* out, int out_dtype, void* stream) {
  const fp4attn_status st = check_directp(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, B, H, N, d,
                                          softmax_scale, affine_a, affine_b, out, out_dtype);
  if (st != FP4ATTN_OK) return st;
  const fp4attn::DirectPArgs a = directp_args(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, B, H, N, d,
                                              softmax_scale, affine_a, affine_b, out, out_dtype);
  return from_hip(fp4attn::launch_forward_mxfp4(a, static_cast<hipStream_t>(stream)), "forward launch");
}

void fp4attn_forward_options_init(fp4attn_forward_options* opts) {
  if (opts != nullptr) *opts = default_options();
}

fp4attn_status fp4attn_forward_mxfp4_ex(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                                        const uint8_t* k_scales, const uint8_t* vt_codes, const uint8_t* vt_scales,
                                        int64_t B, int64_t H, int64_t N, int64_t d, float softmax_scale,
                                        const fp4attn_forward_options* opts, void* out, int out_dtype,
                                        void* stream) {
  fp4attn_forward_options o;
  fp4attn_status st = check_options(opts, &o);
  if (st != FP4ATTN_OK) return st;
  st = check_directp(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, B, H, N, d, softmax_scale,
                     o.affine_a, o.affine_b, out, out_dtype);
  if (st != FP4ATTN_OK) return st;
  fp4attn::DirectPArgs a = directp_args(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, B, H, N, d,
                                        softmax_scale, o.affine_a, o.affine_b, out, out_dtype);
  set_options(a, o);
  return from_hip(fp4attn::launch_forward_mxfp4(a, static_cast<hipStream_t>(stream)), "forward launch");
}

fp4attn_status fp4attn_debug_directp_mxfp4(const uint8_t* q_codes, const uint8_t* q_scales, const uint8_t* k_codes,
                                           const uint8_t* k_scales, const uint8_t* vt_codes,
                                           const uint8_t* vt_scales, int64_t B, int64_t H, int64_t N, int64_t d,
                                           float softmax_scale, const fp4attn_forward_options* opts, void* out,
                                           int out_dtype, const int64_t* row_ids, int64_t n_rows, uint8_t* p_codes,
                                           int16_t* block_exp, int32_t* row_m, float* row_d, uint64_t* wg_clock,
                                           void* stream) {
  fp4attn_forward_options o;
  fp4attn_status st = check_options(opts, &o);
  if (st != FP4ATTN_OK) return st;
  st = check_directp(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, B, H, N, d, softmax_scale,
                     o.affine_a, o.affine_b, out, out_dtype);
  if (st != FP4ATTN_OK) return st;
  if (n_rows < 0 || n_rows > 0x7fffffff) return fail(FP4ATTN_ERR_INVALID_ARG, "n_rows must be in [0, 2^31)");
  if (n_rows > 0) {
    REQUIRE_PTR(row_ids);
    REQUIRE_PTR(p_codes);
    REQUIRE_PTR(block_exp);
    REQUIRE_PTR(row_m);
    REQUIRE_PTR(row_d);
  }
  if (wg_clock != nullptr && (reinterpret_cast<uintptr_t>(wg_clock) & 15) != 0)
    return fail(FP4ATTN_ERR_INVALID_ARG, "wg_clock is not 16-byte aligned");
  fp4attn::DirectPArgs a = directp_args(q_codes, q_scales, k_codes, k_scales, vt_codes, vt_scales, B, H, N, d,
                                        softmax_scale, o.affine_a, o.affine_b, out, out_dtype);
  set_options(a, o);
  a.row_ids = n_rows > 0 ? row_ids : nullptr;
  a.n_rows = (int)n_rows;
  a.p_codes = p_codes;
  a.block_exp = block_exp;
  a.row_m = row_m;
  a.row_d = row_d;
  a.wg_clock = reinterpret_cast<unsigned long long*>(wg_clock);
  return from_hip(fp4attn::launch_forward_mxfp4(a, static_cast<hipStream_t>(stream)), "debug forward launch");
}

fp4attn_status fp4attn_forward_bf16(const void* q, const void* k, const void* v, int64_t B, int64_t H, int64_t N,
                                    int64_t d, float softmax_scale, void* out, int out_dtype, void* stream) {
  REQUIRE_PTR(q);
  REQUIRE_PTR(k);
  REQUIRE_PTR(v);
  REQUIRE_PTR(out);
  const fp4attn_status st = check_attention_shape(B, H, N, d, softmax_scale, out_dtype);
  if (st != FP4ATTN_OK) return st;
  fp4attn::Bf16Args a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.B = (int)B;
  a.H = (int)H;
  a.N = (int)N;
  a.d = (int)d;
  a.out_bf16 = out_dtype == FP4ATTN_BF16;
  a.softmax_scale = softmax_scale;
  return from_hip(fp4attn::launch_forward_bf16(a, static_cast<hipStream_t>(stream)), "bf16 forward launch");
}

fp4attn_status fp4attn_debug_mfma_stream(const uint8_t* a_codes, const uint8_t* b_codes, int blocks, int iters,
                                         float* out, void* stream) {
  REQUIRE_PTR(a_codes);
  REQUIRE_PTR(b_codes);
  REQUIRE_PTR(out);
  if (blocks < 1 || blocks > 65535 || iters < 1)
    return fail(FP4ATTN_ERR_INVALID_ARG, "blocks must be in [1, 65535] and iters >= 1");
  return from_hip(fp4attn::launch_mfma_stream(a_codes, b_codes, blocks, iters, out, static_cast<hipStream_t>(stream)),
                  "mfma stream launch");
}

const char* fp4attn_status_string(int status) {
  switch (status) {
    case FP4ATTN_OK: return "ok";
    case FP4ATTN_ERR_INVALID_ARG: return "invalid argument";
    case FP4ATTN_ERR_UNSUPPORTED: return "unsupported configuration";
    case FP4ATTN_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* fp4attn_last_error(void) { return g_last_error; }

int fp4attn_abi_version(void) { return (2 << 16) | 0; }

}  // extern "C"
