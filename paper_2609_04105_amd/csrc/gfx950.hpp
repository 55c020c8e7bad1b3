// gfx950 (CDNA4) device helpers shared by the HIP kernels of this library.
//
// Operand layouts of the matrix instructions used here (verified on MI355X):
//
//  v_mfma_scale_f32_32x32x64_f8f6f4 with FP4 (E2M1) A and B, C/D fp32 32x32:
//    A (32 x 64):  lane l holds row l % 32, k = 32 * (l / 32) + [0, 32) as 16
//                  bytes, element k in nibble k % 2 of byte k / 2 (low nibble
//                  first); its E8M0 scale is byte OPSEL_A of the lane's scale
//                  register and covers exactly those 32 values.
//    B (64 x 32):  lane l holds column l % 32, k = 32 * (l / 32) + [0, 32),
//                  same packing; scale byte OPSEL_B.
//    C (32 x 32):  lane l, register r holds row 8 (r / 4) + 4 (l / 32) + r % 4,
//                  column l % 32.
//  v_mfma_f32_32x32x16_bf16: A lane l row l % 32, k = 8 (l / 32) + [0, 8);
//    B lane l column l % 32, same k; C as above.
//  v_cvt_scalef32_pk_fp4_f32(old, a, b, scale, sel): byte `sel` of `old`
//    becomes {E2M1(b / scale), E2M1(a / scale)} (a in the low nibble), rounding
//    to nearest even and saturating at 6.
//  v_permlane32_swap(a, b): a's lanes 32..63 and b's lanes 0..31 trade values.
//  v_mfma_scale_f32_32x32x64_f8f6f4 / 16x16x128 with FP8 (E4M3) A and B: the
//    same lane/row/k assignment with one byte per element (32 bytes per lane).
//    (Mixing FP4 with FP8 changes the FP4 operand's k order; not used here.)
//  v_cvt_scalef32_pk_fp8_f32: E4M3 by round to nearest even, subnormals kept;
//    above the E4M3 rounding range the result is NaN, not saturated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <utility>

namespace fp4attn {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef short v8s __attribute__((ext_vector_type(8)));

// E2M1 format selector of the f8f6f4 matrix instructions.
constexpr int kFmtFp4 = 4;

// D = A * B + C on the scaled FP4 matrix unit, 32x32x64.
template <int OPSEL_A, int OPSEL_B>
__device__ __forceinline__ v16f mfma_fp4_32x32x64(v4i a, v4i b, v16f c, int scale_a, int scale_b) {
  v8i a8 = {a[0], a[1], a[2], a[3], 0, 0, 0, 0};
  v8i b8 = {b[0], b[1], b[2], b[3], 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, kFmtFp4, kFmtFp4, OPSEL_A, scale_a,
                                                          OPSEL_B, scale_b);
}

// D = A * B + C on the scaled FP4 matrix unit, 16x16x128 (A lane l: row l % 16,
// k = 32 (l / 16) + [0, 32); B lane l: column l % 16, same k; C lane l, register
// r: row 4 (l / 16) + r, column l % 16).
template <int OPSEL_A, int OPSEL_B>
__device__ __forceinline__ v4f mfma_fp4_16x16x128(v4i a, v4i b, v4f c, int scale_a, int scale_b) {
  v8i a8 = {a[0], a[1], a[2], a[3], 0, 0, 0, 0};
  v8i b8 = {b[0], b[1], b[2], b[3], 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a8, b8, c, kFmtFp4, kFmtFp4, OPSEL_A, scale_a,
                                                           OPSEL_B, scale_b);
}

// E4M3 format selector of the f8f6f4 matrix instructions.
constexpr int kFmtFp8 = 0;

// D = A * B + C on the scaled FP8 (E4M3) matrix unit, 32x32x64 (A lane l: row
// l % 32, k = 32 (l / 32) + [0, 32) as 32 bytes; B likewise by column).
template <int OPSEL_A, int OPSEL_B>
__device__ __forceinline__ v16f mfma_fp8_32x32x64(v8i a, v8i b, v16f c, int scale_a, int scale_b) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, kFmtFp8, kFmtFp8, OPSEL_A, scale_a, OPSEL_B,
                                                          scale_b);
}

// D = A * B + C on the scaled FP8 (E4M3) matrix unit, 16x16x128 (A lane l: row
// l % 16, k = 32 (l / 16) + [0, 32); B likewise by column).
template <int OPSEL_A, int OPSEL_B>
__device__ __forceinline__ v4f mfma_fp8_16x16x128(v8i a, v8i b, v4f c, int scale_a, int scale_b) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, kFmtFp8, kFmtFp8, OPSEL_A, scale_a, OPSEL_B,
                                                           scale_b);
}

// Two fp32 values -> two E4M3 bytes (RNE; inputs must stay below the E4M3
// overflow threshold, where the converter gives NaN), written into the low
// (HI = false) or high 16 bits of `old`.
template <bool HI>
__device__ __forceinline__ unsigned cvt_pk_fp8(unsigned old, float lo, float hi) {
  typedef short v2s __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(__builtin_bit_cast(v2s, old), lo, hi,
                                                                                1.0f, HI));
}

// Value of `v` in lane `src` (any lane), through the LDS crossbar.
__device__ __forceinline__ float lane_read(float v, int src) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src * 4, __builtin_bit_cast(int, v)));
}
__device__ __forceinline__ int lane_read(int v, int src) { return __builtin_amdgcn_ds_bpermute(src * 4, v); }

__device__ __forceinline__ v16f mfma_bf16_32x32x16(v4i a, v4i b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0, 0,
                                                 0);
}

// Two fp32 values -> one byte of E2M1 codes, written into byte SEL of `old`.
template <int SEL>
__device__ __forceinline__ unsigned cvt_pk_fp4(unsigned old, float lo, float hi, float scale) {
  return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, lo, hi, scale, SEL);
}

// Exchange across the two 32-lane halves of the wave (see the header comment).
__device__ __forceinline__ void swap_halves(unsigned& a, unsigned& b) {
  auto r = __builtin_amdgcn_permlane32_swap(a, b, false, false);
  a = r[0];
  b = r[1];
}

__device__ __forceinline__ float as_float(unsigned u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ unsigned as_uint(float f) { return __builtin_bit_cast(unsigned, f); }

// Compile-time loop: f(std::integral_constant<int, I>) for I in [0, N).
template <int N, class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl<N>(f, std::make_integer_sequence<int, N>{});
}

// Workgroup index remapped so that consecutive logical tiles share one of the
// eight XCDs (the hardware deals workgroups to XCDs round-robin).
__device__ __forceinline__ int xcd_remap(int lin, int total) {
  if (total % 8) return lin;
  return (lin % 8) * (total / 8) + lin / 8;
}

}  // namespace fp4attn
