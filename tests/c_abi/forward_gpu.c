/*
 * Plain C99 GPU client of include/fp4attn.h: device buffers from the HIP runtime
 * API, bf16 inputs written on the host, then fp4attn_quantize_mxfp4 (Q, K along
 * d, V along the sequence), fp4attn_forward_mxfp4 and fp4attn_forward_bf16 on
 * one stream.  V is 2^-3 everywhere, which MXFP4 and bf16 represent exactly, so
 * every output element equals 0.125 up to fp32 summation whatever Q and K are
 * (the probabilities sum to one by construction).  Exit status 0 = all held.
 */
#include <math.h>
#include <string.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "fp4attn.h"

enum { B = 1, H = 2, N = 512, D = 128 };

static uint16_t to_bf16(float x) {  /* round to nearest even; inputs are finite */
  uint32_t u;
  memcpy(&u, &x, 4);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

#define HIP_OK(call)                                                   \
  do {                                                                 \
    if ((call) != hipSuccess) {                                        \
      fprintf(stderr, "%s failed\n", #call);                           \
      return 10;                                                       \
    }                                                                  \
  } while (0)

int main(void) {
  const size_t n = (size_t)B * H * N * D;
  uint16_t* host = malloc(3 * n * sizeof(uint16_t));
  float* out = malloc(n * sizeof(float));
  if (!host || !out) return 11;
  uint32_t s = 12345u;
  for (size_t i = 0; i < 2 * n; ++i) {  /* Q, K: uniform in [-2, 2) from a 32-bit LCG */
    s = s * 1664525u + 1013904223u;
    host[i] = to_bf16(((float)(s >> 8) / 16777216.0f) * 4.0f - 2.0f);
  }
  for (size_t i = 2 * n; i < 3 * n; ++i) host[i] = to_bf16(0.125f);

  void *q, *k, *v, *o;
  uint8_t *qc, *qs, *kc, *ks, *vc, *vs;
  HIP_OK(hipMalloc(&q, 3 * n * 2));
  k = (uint8_t*)q + n * 2;
  v = (uint8_t*)q + 2 * n * 2;
  HIP_OK(hipMalloc(&o, n * 4));
  HIP_OK(hipMalloc((void**)&qc, 3 * (n / 2 + n / 32)));
  qs = qc + n / 2;
  kc = qs + n / 32;
  ks = kc + n / 2;
  vc = ks + n / 32;
  vs = vc + n / 2;
  hipStream_t st;
  HIP_OK(hipStreamCreate(&st));
  HIP_OK(hipMemcpy(q, host, 3 * n * 2, hipMemcpyHostToDevice));

  if (fp4attn_quantize_mxfp4(q, FP4ATTN_BF16, B * H, N, D, 1, qc, qs, st) != FP4ATTN_OK) return 1;
  if (fp4attn_quantize_mxfp4(k, FP4ATTN_BF16, B * H, N, D, 1, kc, ks, st) != FP4ATTN_OK) return 2;
  if (fp4attn_quantize_mxfp4(v, FP4ATTN_BF16, B * H, N, D, 0, vc, vs, st) != FP4ATTN_OK) return 3;
  const float scale = 1.0f / sqrtf((float)D);
  for (int route = 0; route < 2; ++route) {
    const fp4attn_status r =
        route == 0 ? fp4attn_forward_mxfp4(qc, qs, kc, ks, vc, vs, B, H, N, D, scale, 1.5f, 1.2f, o, FP4ATTN_F32, st)
                   : fp4attn_forward_bf16(q, k, v, B, H, N, D, scale, o, FP4ATTN_F32, st);
    if (r != FP4ATTN_OK) {
      fprintf(stderr, "route %d: %s (%s)\n", route, fp4attn_status_string(r), fp4attn_last_error());
      return 4 + route;
    }
    HIP_OK(hipStreamSynchronize(st));
    HIP_OK(hipMemcpy(out, o, n * 4, hipMemcpyDeviceToHost));
    double worst = 0.0;
    for (size_t i = 0; i < n; ++i) worst = fmax(worst, fabs((double)out[i] - 0.125));
    printf("route %s: max |O - 0.125| = %.3e\n", route == 0 ? "mxfp4" : "bf16", worst);
    if (!(worst <= 0.125 * 1e-5)) return 6 + route;
  }
  HIP_OK(hipStreamDestroy(st));
  HIP_OK(hipFree(qc));
  HIP_OK(hipFree(o));
  HIP_OK(hipFree(q));
  free(host);
  free(out);
  printf("c-abi forward: all checks held\n");
  return 0;
}
