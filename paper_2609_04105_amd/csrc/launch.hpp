// Host-side launchers of the HIP kernels.  Arguments are already validated by
// the C-ABI layer (api.hip); each launcher only enqueues and reports the launch
// status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fp4attn {

// n_anchor > 0: rows are read in anchor order (rows % n_anchor == 0).
hipError_t launch_quantize_mxfp4(const void* src, int src_dtype, int64_t batch, int64_t rows, int64_t cols, int axis,
                                 int64_t n_anchor, uint8_t* codes, uint8_t* scales, hipStream_t stream);

hipError_t launch_quantize_mxfp8(const void* src, int src_dtype, int64_t batch, int64_t rows, int64_t cols, int axis,
                                 uint8_t* codes, uint8_t* scales, hipStream_t stream);

struct DirectPArgs {
  const uint8_t* q_codes;
  const uint8_t* q_scales;
  const uint8_t* k_codes;
  const uint8_t* k_scales;
  const uint8_t* vt_codes;
  const uint8_t* vt_scales;
  void* out;
  int B, H, N, d;
  int out_bf16;
  float softmax_scale, affine_a, affine_b;
  int ex2_pairs;  // pairs of 16 per 32-key block that take the native exponential
  int guard;      // sampled anchor reference (Alg. 3) instead of the online one
  int guard_margin, guard_shift;
  int causal;     // query i sees keys j <= i
  int pv_fp8;     // P and V as FP8 (E4M3) payloads; V operands are MXFP8
  float* lse;     // optional [B, H, N] natural-log row normaliser
  // test hook (all null / zero for the plain forward)
  const int64_t* row_ids;
  int n_rows;
  uint8_t* p_codes;
  int16_t* block_exp;
  int32_t* row_m;
  float* row_d;
  unsigned long long* wg_clock;  // may be null
};

hipError_t launch_forward_mxfp4(const DirectPArgs& a, hipStream_t stream);

struct Bf16Args {
  const void* q;
  const void* k;
  const void* v;
  void* out;
  int B, H, N, d;
  int out_bf16;
  float softmax_scale;
};

hipError_t launch_forward_bf16(const Bf16Args& a, hipStream_t stream);

}  // namespace fp4attn
