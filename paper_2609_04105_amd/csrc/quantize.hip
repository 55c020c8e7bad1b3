// MXFP4 and MXFP8 input quantizers.
//
// Quantizer (eq. mx-scale): per block of 32 values with absolute maximum a,
// the E8M0 amplitude is 2^floor(log2 a) or 2^ceil(log2 a), whichever has the
// smaller squared reconstruction error (ties keep the ceiling).  With
// r = 6|v| / 2^e_ceil, ceiling codes qc = E2M1(r) and floor codes qf = E2M1(2r),
// the floor wins iff sum (2 qc - qf)(4 r - qf - 2 qc) < 0; every term of that
// sum is exact in fp64 for fp32/bf16 inputs, so the choice is exact.
// bf16 inputs take a 32-bit path with the hardware E2M1 converter (exact too,
// see mxfp4_block_bf16), 16-byte loads for Q and K and two columns per thread
// for V^T; fp32 inputs and odd shapes take the fp64 kernel.  One thread owns
// one block (bf16 V^T: one block of each of two columns).
#include "gfx950.hpp"
#include "launch.hpp"

namespace fp4attn {

typedef float v2f __attribute__((ext_vector_type(2)));


// Index k of the E2M1 magnitude {0, .5, 1, 1.5, 2, 3, 4, 6} nearest to r >= 0,
// ties to even k, saturating: count the boundaries at or below r, each tie
// counted toward the even neighbour.
__device__ __forceinline__ int e2m1_index(double r) {
  return (r > 0.25) + (r >= 0.75) + (r > 1.25) + (r >= 1.75) + (r > 2.5) + (r >= 3.5) + (r > 5.0);
}
__device__ __forceinline__ double e2m1_value(int k) {
  // 0, .5, 1, 1.5 for k < 4; 2, 3, 4, 6 for k >= 4
  return k < 4 ? 0.5 * k : (k == 7 ? 6.0 : (double)(k - 2));
}

template <typename T>
__device__ __forceinline__ float load_as_float(const T* p);
template <>
__device__ __forceinline__ float load_as_float<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_as_float<uint16_t>(const uint16_t* p) {
  return __builtin_bit_cast(float, (unsigned)(*p) << 16);
}

// Source row of row r of the anchor-ordered matrix (Sec. "Fix 3": the anchor
// rows j * stride, j < n_anchor, first, then every other row in order);
// stride 0 is the identity.  Always within [0, n_anchor * stride).
__device__ __forceinline__ int64_t anchor_source_row(int64_t r, int64_t n_anchor, int64_t stride) {
  if (stride <= 1) return r;
  if (r < n_anchor) return r * stride;
  const int64_t k = r - n_anchor;
  return (k / (stride - 1)) * stride + 1 + k % (stride - 1);
}

// axis == 1: blocks along the contiguous axis (Q, K).  axis == 0: blocks along
// rows, output transposed (V).  Rows are read in anchor order when
// anchor_stride > 0.
template <typename T, int AXIS>
__global__ __launch_bounds__(256) void quantize_mxfp4_kernel(const T* __restrict__ src, int64_t batch, int64_t rows,
                                                             int64_t cols, uint8_t* __restrict__ codes,
                                                             uint8_t* __restrict__ scales, int64_t n_anchor,
                                                             int64_t anchor_stride) {
  const int64_t nblk = AXIS == 1 ? cols / 32 : rows / 32;
  const int64_t outer = AXIS == 1 ? rows : cols;
  const int64_t total = batch * outer * nblk;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  int64_t b, o, blk;
  if (AXIS == 1) {  // consecutive threads take consecutive blocks of one row
    blk = t % nblk;
    o = (t / nblk) % outer;
    b = t / (nblk * outer);
  } else {  // consecutive threads take consecutive columns: coalesced loads
    o = t % outer;
    blk = (t / outer) % nblk;
    b = t / (outer * nblk);
  }
  float v[32];
  if (AXIS == 1) {
    const T* p = src + (b * rows + anchor_source_row(o, n_anchor, anchor_stride)) * cols + blk * 32;
#pragma unroll
    for (int j = 0; j < 32; ++j) v[j] = load_as_float<T>(p + j);
  } else if (anchor_stride <= 1) {
    const T* p = src + (b * rows + blk * 32) * cols + o;
#pragma unroll
    for (int j = 0; j < 32; ++j) v[j] = load_as_float<T>(p + (int64_t)j * cols);
  } else {
    const T* p = src + b * rows * cols + o;
#pragma unroll
    for (int j = 0; j < 32; ++j) v[j] = load_as_float<T>(p + anchor_source_row(blk * 32 + j, n_anchor, anchor_stride) * cols);
  }
  float amax = 0.0f;
  bool finite = true;
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    finite = finite && __builtin_isfinite(v[j]);
    amax = fmaxf(amax, fabsf(v[j]));
  }
  int e = 0;
  unsigned ubyte;
  if (!finite) {
    ubyte = 255;
  } else if (amax == 0.0f) {
    ubyte = 0;
  } else {
    int x;
    const float m = frexpf(amax, &x);  // amax = m 2^x, m in [0.5, 1)
    const int e_floor = x - 1;
    const int e_ceil = (m == 0.5f) ? x - 1 : x;
    double delta = 0.0;
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const double r = ldexp(6.0 * (double)fabsf(v[j]), -e_ceil);
      const double qc = e2m1_value(e2m1_index(r));
      const double qf = e2m1_value(e2m1_index(2.0 * r));
      delta += (2.0 * qc - qf) * (4.0 * r - qf - 2.0 * qc);
    }
    e = (e_floor != e_ceil && delta < 0.0) ? e_floor : e_ceil;
    e = e < -127 ? -127 : (e > 127 ? 127 : e);
    ubyte = (unsigned)(e + 127);
  }
  unsigned w[4] = {0u, 0u, 0u, 0u};
  if (finite) {
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const int k = e2m1_index(ldexp(6.0 * (double)fabsf(v[j]), -e));
      const unsigned code = (unsigned)k | (__builtin_signbit(v[j]) ? 8u : 0u);
      w[j / 8] |= code << (4 * (j % 8));
    }
  }
  uint8_t* cdst = codes + (b * outer + o) * (nblk * 16) + blk * 16;
  *reinterpret_cast<v4i*>(cdst) = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
  scales[(b * outer + o) * nblk + blk] = (uint8_t)ubyte;
}

// bf16 fast path of the same rule, exact in 32-bit arithmetic.  A bf16 value
// has at most 8 significant bits, so r = 6 v / 2^e_ceil has at most 10 and is
// exact in fp32; the hardware converter's E2M1 rounding (nearest, ties to the
// even code, saturating at 6) gives qc = E2M1(r) and qf = E2M1(2 r) exactly and
// the decode instruction returns their values, so the rule's sum is evaluated
// exactly (see below).  The codes of the chosen amplitude are the ones already
// converted (unless the E8M0 range clamps it).
//   raw[i]: elements 2i (bits 0-15) and 2i + 1 (bits 16-31).  Returns the E8M0
//   byte; codes[j] holds elements 8 j .. 8 j + 7, even element in the low nibble.
__device__ __forceinline__ unsigned mxfp4_block_bf16(const unsigned (&raw)[16], unsigned (&codes)[4]) {
  // Block maximum on the magnitude bits, two bf16 values per packed 16-bit max:
  // magnitudes order as their bit patterns, and Inf and NaN sort above every
  // finite value.
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  u16x2 mx = {0, 0};
#pragma unroll
  for (int i = 0; i < 16; ++i) mx = __builtin_elementwise_max(mx, __builtin_bit_cast(u16x2, raw[i] & 0x7fff7fffu));
  const unsigned amax_bits = mx[0] > mx[1] ? mx[0] : mx[1];
  if (amax_bits >= 0x7f80u) {  // a NaN or an infinity in the block
#pragma unroll
    for (int j = 0; j < 4; ++j) codes[j] = 0u;
    return 255u;
  }
  // Signed values go straight into the converter: its codes carry the input's
  // sign bit (-0.0 and negative values that round to zero give 0x8).
  // encode: the codes of 6 v / 2^e, scaled in two exact steps (valid for every
  // E8M0 exponent, where the single factor 6 / 2^e may overflow).
  auto encode = [&](int e, unsigned (&w)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      unsigned acc = 0u;
      static_for<4>([&](auto P_) {
        constexpr int pb = decltype(P_)::value;
        const unsigned word = raw[4 * j + pb];
        const float v0 = __builtin_bit_cast(float, word << 16), v1 = __builtin_bit_cast(float, word & 0xffff0000u);
        acc = cvt_pk_fp4<pb>(pb == 0 ? 0u : acc, 6.0f * ldexpf(v0, -e), 6.0f * ldexpf(v1, -e), 1.0f);
      });
      w[j] = acc;
    }
  };
  if (amax_bits == 0u) {  // zero block: byte 0, every code a signed zero
    encode(0, codes);
    return 0u;
  }
  int x;
  const float m = frexpf(__builtin_bit_cast(float, amax_bits << 16), &x);  // amax = m 2^x, m in [0.5, 1)
  const int e_floor = x - 1, e_ceil = (m == 0.5f) ? x - 1 : x;
  // r = 6 v / 2^e_ceil (one exact multiply), qc = E2M1(r) and qf = E2M1(2 r)
  // (the converter divides by its scale operand and saturates at 6).  The
  // choice compares 4 sum(a r) with sum(a b), a = 2 qc - qf, b = 2 qc + qf: the
  // floor amplitude wins iff sum a (4 r - b) < 0.  Only values with |r| >= 1/8
  // have a != 0; such r are multiples of 2^-12, and |a| <= qc <= 6 because
  // qf >= qc, so both sums are exact in fp32 (multiples of 2^-13 below 2^11, and
  // of 2^-2 below 2^12).
  // The single factor 6 / 2^e_ceil is finite for e_ceil >= -125; blocks below
  // that (amax under 2^-125) take the two-step scaling of encode.
  const float sc = ldexpf(6.0f, -e_ceil);
  unsigned cc[4], cf[4];
  float s_ar = 0.0f, s_ab = 0.0f;
  auto convert = [&](auto TWO_STEP_) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      unsigned wc = 0u, wf = 0u;
      static_for<4>([&](auto P_) {
        constexpr int pb = decltype(P_)::value;
        const unsigned word = raw[4 * j + pb];
        const float v0 = __builtin_bit_cast(float, word << 16), v1 = __builtin_bit_cast(float, word & 0xffff0000u);
        float r0, r1;
        if constexpr (decltype(TWO_STEP_)::value) {
          r0 = 6.0f * ldexpf(v0, -e_ceil);
          r1 = 6.0f * ldexpf(v1, -e_ceil);
        } else {
          r0 = v0 * sc;
          r1 = v1 * sc;
        }
        wc = cvt_pk_fp4<pb>(pb == 0 ? 0u : wc, r0, r1, 1.0f);
        wf = cvt_pk_fp4<pb>(pb == 0 ? 0u : wf, r0, r1, 0.5f);
        const v2f qc = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wc, 1.0f, pb);
        const v2f qf = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wf, 1.0f, pb);
        const float a0 = fmaf(2.0f, qc[0], -qf[0]), a1 = fmaf(2.0f, qc[1], -qf[1]);
        s_ar = fmaf(a1, r1, fmaf(a0, r0, s_ar));
        s_ab = fmaf(a1, fmaf(2.0f, qc[1], qf[1]), fmaf(a0, fmaf(2.0f, qc[0], qf[0]), s_ab));
      });
      cc[j] = wc;
      cf[j] = wf;
    }
  };
  if (e_ceil >= -125) convert(std::false_type{});
  else convert(std::true_type{});
  int e = (e_floor != e_ceil && 4.0f * s_ar < s_ab) ? e_floor : e_ceil;
  e = e < -127 ? -127 : (e > 127 ? 127 : e);
  if (e == e_ceil) {
#pragma unroll
    for (int j = 0; j < 4; ++j) codes[j] = cc[j];
  } else if (e == e_floor) {
#pragma unroll
    for (int j = 0; j < 4; ++j) codes[j] = cf[j];
  } else {  // amplitude clamped to the E8M0 range
    encode(e, codes);
  }
  return (unsigned)(e + 127);
}

// bf16, blocks along the contiguous axis (Q, K): one block per thread, four
// 16-byte loads.
__global__ __launch_bounds__(256) void quantize_mxfp4_bf16_rows_kernel(const uint16_t* __restrict__ src, int64_t batch,
                                                                       int64_t rows, int64_t cols,
                                                                       uint8_t* __restrict__ codes,
                                                                       uint8_t* __restrict__ scales, int64_t n_anchor,
                                                                       int64_t anchor_stride) {
  const int64_t nblk = cols / 32;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= batch * rows * nblk) return;
  const int64_t blk = t % nblk, o = (t / nblk) % rows, b = t / (nblk * rows);
  const uint4* p = reinterpret_cast<const uint4*>(src + (b * rows + anchor_source_row(o, n_anchor, anchor_stride)) * cols +
                                                  blk * 32);
  unsigned raw[16];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint4 q = p[i];
    raw[4 * i] = q.x;
    raw[4 * i + 1] = q.y;
    raw[4 * i + 2] = q.z;
    raw[4 * i + 3] = q.w;
  }
  unsigned w[4];
  const unsigned u = mxfp4_block_bf16(raw, w);
  *reinterpret_cast<v4i*>(codes + t * 16) = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
  scales[t] = (uint8_t)u;
}

// bf16, blocks along rows with transposed output (V): a thread takes one block
// of two adjacent columns (one 4-byte load per row; a wave reads 256-byte row
// segments).  cols % 2 == 0.  (Several blocks per thread, for longer runs of
// contiguous code bytes, measured slower: fewer waves in flight.)
__global__ __launch_bounds__(256) void quantize_mxfp4_bf16_cols_kernel(const uint16_t* __restrict__ src, int64_t batch,
                                                                       int64_t rows, int64_t cols,
                                                                       uint8_t* __restrict__ codes,
                                                                       uint8_t* __restrict__ scales, int64_t n_anchor,
                                                                       int64_t anchor_stride) {
  const int64_t nblk = rows / 32, npair = cols / 2;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= batch * nblk * npair) return;
  const int64_t cp = t % npair, blk = (t / npair) % nblk, b = t / (npair * nblk);
  const uint16_t* base = src + b * rows * cols + 2 * cp;
  unsigned pair[32];
#pragma unroll
  for (int j = 0; j < 32; ++j)
    pair[j] = *reinterpret_cast<const unsigned*>(base + anchor_source_row(blk * 32 + j, n_anchor, anchor_stride) * cols);
  unsigned raw0[16], raw1[16];  // column 2 cp and 2 cp + 1, rows in order
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    raw0[i] = (pair[2 * i] & 0xffffu) | (pair[2 * i + 1] << 16);
    raw1[i] = (pair[2 * i] >> 16) | (pair[2 * i + 1] & 0xffff0000u);
  }
  const int64_t col0 = b * cols + 2 * cp;
  unsigned w[4];
  scales[col0 * nblk + blk] = (uint8_t)mxfp4_block_bf16(raw0, w);
  *reinterpret_cast<v4i*>(codes + (col0 * nblk + blk) * 16) = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
  scales[(col0 + 1) * nblk + blk] = (uint8_t)mxfp4_block_bf16(raw1, w);
  *reinterpret_cast<v4i*>(codes + ((col0 + 1) * nblk + blk) * 16) = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
}

// The E8M0 bytes of blocks 8 grp .. 8 grp + 7 of one column (byte l of `run` is
// block 8 grp + l) to `dst`: one 8-byte store when every column has whole groups
// of 8 blocks (dst is then 8-byte aligned), else one byte per block that exists.
__device__ __forceinline__ void store_scale_run(uint8_t* dst, uint2 run, int64_t nblk, int64_t grp) {
  if (nblk % 8 == 0) {
    *reinterpret_cast<uint2*>(dst) = run;
  } else {
    const uint64_t bytes = ((uint64_t)run.y << 32) | run.x;
    for (int l = 0; l < 8 && grp * 8 + l < nblk; ++l) dst[l] = (uint8_t)(bytes >> (8 * l));
  }
}

// bf16, blocks along rows with transposed output (V), staged: a workgroup takes
// 64 columns x 256 rows (32 column pairs x 8 blocks; a thread quantizes one block
// of two adjacent columns as above), parks its codes and scale bytes in LDS, and
// writes each column's 8 blocks of codes as one contiguous 128-byte run (each
// store instruction of a wave covers 64 contiguous bytes of 16 columns) and its 8
// scale bytes with one store.  The loads stay 128-byte row segments; the
// workgroups that take the column groups of the same rows are launched next to
// each other, so the wider rows of d = 128 are read whole at about the same
// time.  cols % 64 == 0; blocks past the last are skipped (their threads still
// meet the barrier).
__global__ __launch_bounds__(256) void quantize_mxfp4_bf16_cols_staged_kernel(
    const uint16_t* __restrict__ src, int64_t batch, int64_t rows, int64_t cols, uint8_t* __restrict__ codes,
    uint8_t* __restrict__ scales, int64_t n_anchor, int64_t anchor_stride) {
  __shared__ uint4 code_lds[64][8];
  __shared__ uint2 scale_lds[64];  // 8 bytes per column
  const int64_t nblk = rows / 32, ngrp = (nblk + 7) / 8, ncg = cols / 64;
  const int64_t cg = blockIdx.x % ncg, grp = (blockIdx.x / ncg) % ngrp, b = blockIdx.x / (ngrp * ncg);
  const int tid = threadIdx.x, cp = tid % 32, lb = tid / 32;
  const int64_t blk = grp * 8 + lb;
  if (blk < nblk) {
    const uint16_t* base = src + b * rows * cols + cg * 64 + 2 * cp;
    unsigned pair[32];
#pragma unroll
    for (int j = 0; j < 32; ++j)
      pair[j] = *reinterpret_cast<const unsigned*>(base + anchor_source_row(blk * 32 + j, n_anchor, anchor_stride) * cols);
    unsigned raw0[16], raw1[16];  // column 2 cp and 2 cp + 1, rows in order
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      raw0[i] = (pair[2 * i] & 0xffffu) | (pair[2 * i + 1] << 16);
      raw1[i] = (pair[2 * i] >> 16) | (pair[2 * i + 1] & 0xffff0000u);
    }
    unsigned w[4];
    uint8_t* sb = reinterpret_cast<uint8_t*>(scale_lds);
    sb[16 * cp + lb] = (uint8_t)mxfp4_block_bf16(raw0, w);
    code_lds[2 * cp][lb] = uint4{w[0], w[1], w[2], w[3]};
    sb[16 * cp + 8 + lb] = (uint8_t)mxfp4_block_bf16(raw1, w);
    code_lds[2 * cp + 1][lb] = uint4{w[0], w[1], w[2], w[3]};
  }
  __syncthreads();
  // thread t writes blocks (t % 4) and (t % 4) + 4 of column t / 4
  const int c = tid / 4, part = tid % 4;
  const int64_t col = b * cols + cg * 64 + c;
  uint8_t* cdst = codes + (col * nblk + grp * 8) * 16;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int l = part + 4 * k;
    if (grp * 8 + l < nblk) *reinterpret_cast<uint4*>(cdst + l * 16) = code_lds[c][l];
  }
  if (tid < 64) store_scale_run(scales + (b * cols + cg * 64 + tid) * nblk + grp * 8, scale_lds[tid], nblk, grp);
}

// MXFP8 (E4M3 payload + E8M0 per 32 values): the amplitude is the smallest
// power of two 2^e with amax / 2^e <= 448, so no payload saturates; payloads
// are v / 2^e (exact) rounded to nearest even by the hardware converter, which
// keeps E4M3 subnormals.  Zero block: u = 0; non-finite block: u = 255, codes 0.
// Codes are stored one byte per value, in the same orientation as the MXFP4
// quantizer (axis 0: transposed).
// One MXFP8 block: returns the E8M0 byte; w[i] holds the E4M3 payloads of values
// 4 i .. 4 i + 3.
__device__ __forceinline__ unsigned mxfp8_block(const float (&v)[32], unsigned (&w)[8]) {
  float amax = 0.0f;
  bool finite = true;
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    finite = finite && __builtin_isfinite(v[j]);
    amax = fmaxf(amax, fabsf(v[j]));
  }
  unsigned ubyte;
  int e = 0;
  if (!finite) {
    ubyte = 255;
  } else if (amax == 0.0f) {
    ubyte = 0;
  } else {
    int x;
    frexpf(amax, &x);          // amax = m 2^x, m in [0.5, 1)
    e = x - 9;                 // amax / 2^e in [256, 512)
    if (ldexpf(amax, -e) > 448.0f) ++e;
    e = e < -127 ? -127 : (e > 127 ? 127 : e);
    ubyte = (unsigned)(e + 127);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if (finite) {
      const float a0 = ldexpf(v[4 * i], -e), a1 = ldexpf(v[4 * i + 1], -e);
      const float a2 = ldexpf(v[4 * i + 2], -e), a3 = ldexpf(v[4 * i + 3], -e);
      w[i] = cvt_pk_fp8<true>(cvt_pk_fp8<false>(0u, a0, a1), a2, a3);
    } else {
      w[i] = 0u;
    }
  }
  return ubyte;
}

template <typename T, int AXIS>
__global__ __launch_bounds__(256) void quantize_mxfp8_kernel(const T* __restrict__ src, int64_t batch, int64_t rows,
                                                             int64_t cols, uint8_t* __restrict__ codes,
                                                             uint8_t* __restrict__ scales) {
  const int64_t nblk = AXIS == 1 ? cols / 32 : rows / 32;
  const int64_t outer = AXIS == 1 ? rows : cols;
  const int64_t total = batch * outer * nblk;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  int64_t b, o, blk;
  if (AXIS == 1) {
    blk = t % nblk;
    o = (t / nblk) % outer;
    b = t / (nblk * outer);
  } else {
    o = t % outer;
    blk = (t / outer) % nblk;
    b = t / (outer * nblk);
  }
  float v[32];
  if (AXIS == 1) {
    const T* p = src + (b * rows + o) * cols + blk * 32;
#pragma unroll
    for (int j = 0; j < 32; ++j) v[j] = load_as_float<T>(p + j);
  } else {
    const T* p = src + (b * rows + blk * 32) * cols + o;
#pragma unroll
    for (int j = 0; j < 32; ++j) v[j] = load_as_float<T>(p + (int64_t)j * cols);
  }
  unsigned w[8];
  const unsigned ubyte = mxfp8_block(v, w);
  uint8_t* cdst = codes + (b * outer + o) * (nblk * 32) + blk * 32;
  *reinterpret_cast<v4i*>(cdst) = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
  *reinterpret_cast<v4i*>(cdst + 16) = v4i{(int)w[4], (int)w[5], (int)w[6], (int)w[7]};
  scales[(b * outer + o) * nblk + blk] = (uint8_t)ubyte;
}

// MXFP8 of bf16 blocks along rows with transposed output (V of the FP8 P/V
// route), staged like the MXFP4 V^T kernel: a workgroup takes 64 columns x 256
// rows (32 column pairs x 8 blocks, 4-byte row loads), parks its payloads and
// scale bytes in LDS and writes each column's 8 blocks as one 256-byte run (each
// store instruction of a wave covers 64 contiguous bytes of 16 columns) and its
// 8 scale bytes with one store.
// cols % 64 == 0; blocks past the last are skipped (their threads still meet
// the barrier).
__global__ __launch_bounds__(256) void quantize_mxfp8_bf16_cols_staged_kernel(
    const uint16_t* __restrict__ src, int64_t batch, int64_t rows, int64_t cols, uint8_t* __restrict__ codes,
    uint8_t* __restrict__ scales) {
  __shared__ uint4 code_lds[64][16];  // column x 16-byte chunk of its 256-byte run
  __shared__ uint2 scale_lds[64];      // 8 bytes per column
  const int64_t nblk = rows / 32, ngrp = (nblk + 7) / 8, ncg = cols / 64;
  const int64_t cg = blockIdx.x % ncg, grp = (blockIdx.x / ncg) % ngrp, b = blockIdx.x / (ngrp * ncg);
  const int tid = threadIdx.x, cp = tid % 32, lb = tid / 32;
  const int64_t blk = grp * 8 + lb;
  if (blk < nblk) {
    const uint16_t* base = src + (b * rows + blk * 32) * cols + cg * 64 + 2 * cp;
    float v0[32], v1[32];
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const unsigned pr = *reinterpret_cast<const unsigned*>(base + (int64_t)j * cols);
      v0[j] = __builtin_bit_cast(float, pr << 16);
      v1[j] = __builtin_bit_cast(float, pr & 0xffff0000u);
    }
    unsigned w[8];
    uint8_t* sb = reinterpret_cast<uint8_t*>(scale_lds);
    sb[16 * cp + lb] = (uint8_t)mxfp8_block(v0, w);
    code_lds[2 * cp][2 * lb] = uint4{w[0], w[1], w[2], w[3]};
    code_lds[2 * cp][2 * lb + 1] = uint4{w[4], w[5], w[6], w[7]};
    sb[16 * cp + 8 + lb] = (uint8_t)mxfp8_block(v1, w);
    code_lds[2 * cp + 1][2 * lb] = uint4{w[0], w[1], w[2], w[3]};
    code_lds[2 * cp + 1][2 * lb + 1] = uint4{w[4], w[5], w[6], w[7]};
  }
  __syncthreads();
  // thread t writes 16-byte chunks (t % 4) + 4 k, k < 4, of column t / 4 (chunk
  // 2 l + h is half h of block l)
  const int c = tid / 4, part = tid % 4;
  const int64_t col = b * cols + cg * 64 + c;
  uint8_t* cdst = codes + (col * nblk + grp * 8) * 32;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int ch = part + 4 * k;
    if (grp * 8 + ch / 2 < nblk) *reinterpret_cast<uint4*>(cdst + ch * 16) = code_lds[c][ch];
  }
  if (tid < 64) store_scale_run(scales + (b * cols + cg * 64 + tid) * nblk + grp * 8, scale_lds[tid], nblk, grp);
}

hipError_t launch_quantize_mxfp4(const void* src, int src_dtype, int64_t batch, int64_t rows, int64_t cols, int axis,
                                 int64_t n_anchor, uint8_t* codes, uint8_t* scales, hipStream_t stream) {
  const int64_t stride = n_anchor > 0 ? rows / n_anchor : 0;
  const int64_t nblk = axis == 1 ? cols / 32 : rows / 32;
  const int64_t outer = axis == 1 ? rows : cols;
  const int64_t total = batch * outer * nblk;
  const dim3 grid((unsigned)((total + 255) / 256)), block(256);
  if (src_dtype == 1 && axis == 1) {
    hipLaunchKernelGGL(quantize_mxfp4_bf16_rows_kernel, grid, block, 0, stream, (const uint16_t*)src, batch, rows, cols,
                       codes, scales, n_anchor, stride);
    return hipGetLastError();
  }
  if (src_dtype == 1 && axis == 0 && cols % 64 == 0) {
    const int64_t groups = batch * (cols / 64) * ((nblk + 7) / 8);
    hipLaunchKernelGGL(quantize_mxfp4_bf16_cols_staged_kernel, dim3((unsigned)groups), block, 0, stream,
                       (const uint16_t*)src, batch, rows, cols, codes, scales, n_anchor, stride);
    return hipGetLastError();
  }
  if (src_dtype == 1 && axis == 0 && cols % 2 == 0) {
    const int64_t threads = batch * nblk * (cols / 2);
    hipLaunchKernelGGL(quantize_mxfp4_bf16_cols_kernel, dim3((unsigned)((threads + 255) / 256)), block, 0, stream,
                       (const uint16_t*)src, batch, rows, cols, codes, scales, n_anchor, stride);
    return hipGetLastError();
  }
  if (src_dtype == 0) {
    if (axis == 1)
      hipLaunchKernelGGL((quantize_mxfp4_kernel<float, 1>), grid, block, 0, stream, (const float*)src, batch, rows,
                         cols, codes, scales, n_anchor, stride);
    else
      hipLaunchKernelGGL((quantize_mxfp4_kernel<float, 0>), grid, block, 0, stream, (const float*)src, batch, rows,
                         cols, codes, scales, n_anchor, stride);
  } else {
    if (axis == 1)
      hipLaunchKernelGGL((quantize_mxfp4_kernel<uint16_t, 1>), grid, block, 0, stream, (const uint16_t*)src, batch,
                         rows, cols, codes, scales, n_anchor, stride);
    else
      hipLaunchKernelGGL((quantize_mxfp4_kernel<uint16_t, 0>), grid, block, 0, stream, (const uint16_t*)src, batch,
                         rows, cols, codes, scales, n_anchor, stride);
  }
  return hipGetLastError();
}

hipError_t launch_quantize_mxfp8(const void* src, int src_dtype, int64_t batch, int64_t rows, int64_t cols, int axis,
                                 uint8_t* codes, uint8_t* scales, hipStream_t stream) {
  const int64_t nblk = axis == 1 ? cols / 32 : rows / 32;
  const int64_t outer = axis == 1 ? rows : cols;
  const int64_t total = batch * outer * nblk;
  const dim3 grid((unsigned)((total + 255) / 256)), block(256);
  if (src_dtype == 1 && axis == 0 && cols % 64 == 0) {
    const int64_t groups = batch * (cols / 64) * ((nblk + 7) / 8);
    hipLaunchKernelGGL(quantize_mxfp8_bf16_cols_staged_kernel, dim3((unsigned)groups), block, 0, stream,
                       (const uint16_t*)src, batch, rows, cols, codes, scales);
    return hipGetLastError();
  }
  if (src_dtype == 0) {
    if (axis == 1)
      hipLaunchKernelGGL((quantize_mxfp8_kernel<float, 1>), grid, block, 0, stream, (const float*)src, batch, rows,
                         cols, codes, scales);
    else
      hipLaunchKernelGGL((quantize_mxfp8_kernel<float, 0>), grid, block, 0, stream, (const float*)src, batch, rows,
                         cols, codes, scales);
  } else {
    if (axis == 1)
      hipLaunchKernelGGL((quantize_mxfp8_kernel<uint16_t, 1>), grid, block, 0, stream, (const uint16_t*)src, batch,
                         rows, cols, codes, scales);
    else
      hipLaunchKernelGGL((quantize_mxfp8_kernel<uint16_t, 0>), grid, block, 0, stream, (const uint16_t*)src, batch,
                         rows, cols, codes, scales);
  }
  return hipGetLastError();
}

}  // namespace fp4attn
