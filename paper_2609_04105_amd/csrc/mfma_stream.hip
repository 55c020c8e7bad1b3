// Sustained rate of the scaled FP4 matrix unit on given operands: the ceiling
// against which the forward's matrix work is compared.  Each thread keeps four
// A and four B fragments (16 bytes each) of its own in registers and issues
// `iters` rounds of four independent 32x32x64 FP4 products (E8M0 scales 127),
// with nothing else in the loop; it then writes the sum of its accumulators.
#include "gfx950.hpp"

namespace fp4attn {
namespace {

__global__ __launch_bounds__(256) void mfma_stream_kernel(const v4i* __restrict__ a, const v4i* __restrict__ b,
                                                          int iters, float* __restrict__ out) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  v4i fa[4], fb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    fa[i] = a[g * 4 + i];
    fb[i] = b[g * 4 + i];
  }
  v16f acc[4] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = mfma_fp4_32x32x64<0, 0>(fa[i], fb[(i + 1) & 3], acc[i], 127, 127);
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[i][r];
  out[g] = s;
}

}  // namespace

hipError_t launch_mfma_stream(const void* a, const void* b, int blocks, int iters, float* out, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_stream_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<const v4i*>(a),
                     static_cast<const v4i*>(b), iters, out);
  return hipGetLastError();
}

}  // namespace fp4attn
