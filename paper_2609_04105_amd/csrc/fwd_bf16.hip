// Same-design BF16 attention forward: the in-house speed baseline for the
// paper's canonical speedup t_BF16 / t_FP4 (eq. canonical-speedup).
//
// Textbook softmax attention (eq. exact-attention) with the online recurrence
// (eq. online-recurrence) in base 2.  The structure mirrors the MXFP4 kernel:
// transposed products S^T = K Q^T and O^T = V^T P^T on
// v_mfma_f32_32x32x16_bf16 so that lane l owns query l % 32, 32 queries per
// wave, K/V tiles (64 keys) staged in LDS in operand order and double-buffered
// through registers, a lazy rescale that lets the running maximum lag by up to
// 8 binades (exact in fp32), P rounded to bf16 and paired into the PV operand
// with v_permlane32_swap, and the XCD-aware workgroup order.
#include "gfx950.hpp"
#include "launch.hpp"

namespace fp4attn {

namespace {

constexpr int kBN16 = 64;       // keys per LDS tile
constexpr float kTau16 = 8.0f;  // lazy rescale threshold in log2 units
constexpr float kLog2Ef = 1.4426950408889634f;

struct BParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* vt;
  void* out;
  int N, n_qtiles, total;
  float sc;  // softmax_scale * log2(e)
};

template <int D>
struct BLayout {
  static constexpr int kCodes = (kBN16 / 32) * (D / 16) * 1024;  // [sub][d chunk][lane][16 B]
  static constexpr int vCodes = (kBN16 / 16) * (D / 32) * 1024;  // [key chunk][d chunk][lane][16 B]
  static constexpr int kOff = 0;
  static constexpr int vOff = kCodes;
  static constexpr int stage = kCodes + vCodes;
};

template <int D, int NW>
struct BTileRegs {
  static constexpr int NT = NW * 64;
  static constexpr int nK = BLayout<D>::kCodes / 16;
  static constexpr int nV = BLayout<D>::vCodes / 16;
  static constexpr int KPT = (nK + NT - 1) / NT;
  static constexpr int VPT = (nV + NT - 1) / NT;
  v4i k[KPT];
  v4i v[VPT];

  __device__ __forceinline__ void load(const uint16_t* kp, const uint16_t* vtp, int N, int key0, int tid) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int slot = tid + i * NT;
      if (nK % NT == 0 || slot < nK) {
        const int m = slot & 63, rest = slot >> 6;
        const int c = rest % (D / 16), sub = rest / (D / 16);
        const int key = key0 + sub * 32 + (m & 31);
        k[i] = *reinterpret_cast<const v4i*>(kp + (size_t)key * D + 16 * c + 8 * (m >> 5));
      }
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int slot = tid + i * NT;
      if (nV % NT == 0 || slot < nV) {
        const int m = slot & 63, rest = slot >> 6;
        const int cc = rest % (D / 32), kk = rest / (D / 32);
        const int row = 32 * cc + (m & 31);
        v[i] = *reinterpret_cast<const v4i*>(vtp + (size_t)row * N + key0 + 16 * kk + 8 * (m >> 5));
      }
    }
  }
  __device__ __forceinline__ void store(uint8_t* st, int tid) const {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int slot = tid + i * NT;
      if (nK % NT == 0 || slot < nK) *reinterpret_cast<v4i*>(st + BLayout<D>::kOff + slot * 16) = k[i];
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int slot = tid + i * NT;
      if (nV % NT == 0 || slot < nV) *reinterpret_cast<v4i*>(st + BLayout<D>::vOff + slot * 16) = v[i];
    }
  }
};

__device__ __forceinline__ unsigned pack_bf16(float lo, float hi) {
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(unsigned, bf2{(__bf16)lo, (__bf16)hi});
}

template <int D, int NW, bool OUT_BF16>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void fwd_bf16_kernel(const BParams p) {
  using L = BLayout<D>;
  constexpr int BM = NW * 32;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * L::stage];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, h = lane >> 5, lr = lane & 31;
  const int lin = xcd_remap(blockIdx.x, p.total);
  const int bh = lin / p.n_qtiles, qt = lin % p.n_qtiles;
  const int N = p.N;
  const int qrow = qt * BM + wave * 32 + lr;

  const uint16_t* kp = p.k + (size_t)bh * N * D;
  const uint16_t* vtp = p.vt + (size_t)bh * D * N;

  v4i qf[D / 16];
  {
    const uint16_t* qr = p.q + ((size_t)bh * N + qrow) * D;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) qf[c] = *reinterpret_cast<const v4i*>(qr + 16 * c + 8 * h);
  }

  v16f O[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c) O[c] = v16f{};
  float ell = 0.0f;
  float mref = -__builtin_inff();

  BTileRegs<D, NW> regs;
  regs.load(kp, vtp, N, 0, tid);
  regs.store(lds, tid);
  __syncthreads();

  const int ntiles = N / kBN16;
  for (int kt = 0; kt < ntiles; ++kt) {
    uint8_t* st = lds + (kt & 1) * L::stage;
    if (kt + 1 < ntiles) regs.load(kp, vtp, N, (kt + 1) * kBN16, tid);

    v16f S[2];
    static_for<2>([&](auto T_) {
      constexpr int t = decltype(T_)::value;
      v16f a = v16f{};
      static_for<D / 16>([&](auto C_) {
        constexpr int c = decltype(C_)::value;
        const v4i kf = *reinterpret_cast<const v4i*>(st + L::kOff + ((t * (D / 16) + c) * 64 + lane) * 16);
        a = mfma_bf16_32x32x16(kf, qf[c], a);
      });
      S[t] = a;
    });
    float mx = fmaxf(S[0][0], S[1][0]);
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, fmaxf(S[0][r], S[1][r]));
    unsigned xa = as_uint(mx), xb = xa;
    swap_halves(xa, xb);
    const float tmax = fmaxf(as_float(xa), as_float(xb)) * p.sc;
    const bool need = tmax > mref + kTau16;
    if (__builtin_amdgcn_ballot_w64(need)) {
      const float mn = need ? tmax : mref;
      const float alpha = __builtin_amdgcn_exp2f(mref - mn);
#pragma unroll
      for (int c = 0; c < D / 32; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) O[c][r] *= alpha;
      ell *= alpha;
      mref = mn;
    }
    // P = 2^(s * log2 e - m), rounded to bf16 and paired per 16-key chunk.
    v4i P[4];
    static_for<2>([&](auto T_) {
      constexpr int t = decltype(T_)::value;
      static_for<2>([&](auto C_) {
        constexpr int c = decltype(C_)::value;  // 16-key chunk within the 32-key block
        unsigned E[2], F[2];
        static_for<2>([&](auto J_) {
          constexpr int j = decltype(J_)::value;
          const float e0 = __builtin_amdgcn_exp2f(fmaf(S[t][8 * c + 2 * j], p.sc, -mref));
          const float e1 = __builtin_amdgcn_exp2f(fmaf(S[t][8 * c + 2 * j + 1], p.sc, -mref));
          const float f0 = __builtin_amdgcn_exp2f(fmaf(S[t][8 * c + 4 + 2 * j], p.sc, -mref));
          const float f1 = __builtin_amdgcn_exp2f(fmaf(S[t][8 * c + 4 + 2 * j + 1], p.sc, -mref));
          ell += (e0 + e1) + (f0 + f1);
          E[j] = pack_bf16(e0, e1);
          F[j] = pack_bf16(f0, f1);
        });
        swap_halves(E[0], F[0]);
        swap_halves(E[1], F[1]);
        P[2 * t + c] = v4i{(int)E[0], (int)E[1], (int)F[0], (int)F[1]};
      });
    });
    static_for<4>([&](auto KK_) {
      constexpr int kk = decltype(KK_)::value;
      static_for<D / 32>([&](auto C_) {
        constexpr int c = decltype(C_)::value;
        const v4i vf = *reinterpret_cast<const v4i*>(st + L::vOff + ((kk * (D / 32) + c) * 64 + lane) * 16);
        O[c] = mfma_bf16_32x32x16(vf, P[kk], O[c]);
      });
    });

    if (kt + 1 < ntiles) regs.store(lds + ((kt + 1) & 1) * L::stage, tid);
    __syncthreads();
  }

  unsigned la = as_uint(ell), lb = la;
  swap_halves(la, lb);
  const float inv = 1.0f / (as_float(la) + as_float(lb));
  const size_t orow = ((size_t)bh * N + qrow) * D;
#pragma unroll
  for (int c = 0; c < D / 32; ++c) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col = 32 * c + 8 * g + 4 * h;
      const float o0 = O[c][4 * g] * inv, o1 = O[c][4 * g + 1] * inv;
      const float o2 = O[c][4 * g + 2] * inv, o3 = O[c][4 * g + 3] * inv;
      if constexpr (OUT_BF16) {
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(p.out) + orow + col) =
            uint2{pack_bf16(o0, o1), pack_bf16(o2, o3)};
      } else {
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(p.out) + orow + col) = float4{o0, o1, o2, o3};
      }
    }
  }
}

template <int D, int NW>
hipError_t launch_b(const BParams& bp, bool out_bf16, hipStream_t stream) {
  if (out_bf16)
    hipLaunchKernelGGL((fwd_bf16_kernel<D, NW, true>), dim3(bp.total), dim3(NW * 64), 0, stream, bp);
  else
    hipLaunchKernelGGL((fwd_bf16_kernel<D, NW, false>), dim3(bp.total), dim3(NW * 64), 0, stream, bp);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_forward_bf16(const Bf16Args& a, hipStream_t stream) {
  BParams bp{};
  bp.q = static_cast<const uint16_t*>(a.q);
  bp.k = static_cast<const uint16_t*>(a.k);
  bp.vt = static_cast<const uint16_t*>(a.vt);
  bp.out = a.out;
  bp.N = a.N;
  bp.sc = a.softmax_scale * kLog2Ef;
  const int bh = a.B * a.H;
  // the same launch choice as the MXFP4 forward, four-wave tail launch included
  // (B1 N4096: +3 % at H24 and H72, +13 % at H24 d64, -1.6 % at H40)
  const int64_t wide_wgs = a.N % 256 == 0 ? (int64_t)(a.N / 256) * bh : 0;
  const int64_t last_round = wide_wgs % 256;
  const bool tail = wide_wgs > 256 && wide_wgs <= 5 * 256 && last_round != 0 && last_round <= 128;
  const bool wide = wide_wgs >= 256 && !tail;
  const int BM = wide ? 256 : 128;
  bp.n_qtiles = a.N / BM;
  bp.total = bp.n_qtiles * bh;
  if (a.d == 128) return wide ? launch_b<128, 8>(bp, a.out_bf16, stream) : launch_b<128, 4>(bp, a.out_bf16, stream);
  return wide ? launch_b<64, 8>(bp, a.out_bf16, stream) : launch_b<64, 4>(bp, a.out_bf16, stream);
}

}  // namespace fp4attn
