// Direct-P full-MXFP4 attention forward: host dispatch (the kernel and its
// design are in fwd_mxfp4.hpp).  The EX2 = 0 variants are compiled here; the
// native-exponential densities come from fwd_mxfp4_ex2*.hip, the guarded
// variants from fwd_mxfp4_guard.hip and the causal ones from
// fwd_mxfp4_causal.hip, the FP8 P/V route from fwd_mxfp4_fp8pv.hip, all
// compiled in parallel with this file.
#include "fwd_mxfp4.hpp"

namespace fp4attn {
namespace directp_detail {

FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DEFINE, 0, kVarOnline)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 1, kVarOnline)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 2, kVarOnline)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 4, kVarOnline)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 8, kVarOnline)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 16, kVarOnline)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 0, kVarGuard)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 4, kVarGuard)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 16, kVarGuard)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 0, kVarCausal)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 4, kVarCausal)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 16, kVarCausal)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 0, kVarOnline | kPV8)
FP4ATTN_DIRECTP_VARIANTS(FP4ATTN_DIRECTP_DECLARE, 0, kVarCausal | kPV8)

namespace {

// The guarded and causal variants exist for the densities 0, 4 and 16.
template <int D, int NW, bool DUMP, int VAR>
hipError_t dispatch_ex2_subset(const KParams& kp, int ex2, hipStream_t stream) {
  switch (ex2) {
    case 0: return launch_directp<D, NW, DUMP, 0, VAR>(kp, stream);
    case 4: return launch_directp<D, NW, DUMP, 4, VAR>(kp, stream);
    case 16: return launch_directp<D, NW, DUMP, 16, VAR>(kp, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int D, int NW, bool DUMP>
hipError_t dispatch_ex2(const KParams& kp, int ex2, int var, hipStream_t stream) {
  if (var == (kVarOnline | kPV8)) return launch_directp<D, NW, DUMP, 0, kVarOnline | kPV8>(kp, stream);
  if (var == (kVarCausal | kPV8)) return launch_directp<D, NW, DUMP, 0, kVarCausal | kPV8>(kp, stream);
  if (var == kVarGuard) return dispatch_ex2_subset<D, NW, DUMP, kVarGuard>(kp, ex2, stream);
  if (var == kVarCausal) return dispatch_ex2_subset<D, NW, DUMP, kVarCausal>(kp, ex2, stream);
  switch (ex2) {
    case 0: return launch_directp<D, NW, DUMP, 0, kVarOnline>(kp, stream);
    case 1: return launch_directp<D, NW, DUMP, 1, kVarOnline>(kp, stream);
    case 2: return launch_directp<D, NW, DUMP, 2, kVarOnline>(kp, stream);
    case 4: return launch_directp<D, NW, DUMP, 4, kVarOnline>(kp, stream);
    case 8: return launch_directp<D, NW, DUMP, 8, kVarOnline>(kp, stream);
    case 16: return launch_directp<D, NW, DUMP, 16, kVarOnline>(kp, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int D, int NW>
hipError_t dispatch_dump(const KParams& kp, bool dump, int ex2, int var, hipStream_t stream) {
  return dump ? dispatch_ex2<D, NW, true>(kp, ex2, var, stream) : dispatch_ex2<D, NW, false>(kp, ex2, var, stream);
}

}  // namespace
}  // namespace directp_detail

hipError_t launch_forward_mxfp4(const DirectPArgs& a, hipStream_t stream) {
  using namespace directp_detail;
  KParams kp{};
  kp.qc = a.q_codes;
  kp.qs = a.q_scales;
  kp.kc = a.k_codes;
  kp.ks = a.k_scales;
  kp.vc = a.vt_codes;
  kp.vs = a.vt_scales;
  kp.out = a.out;
  kp.N = a.N;
  // fp32 coefficients of the folded code map (see the file header).
  const double s = (double)a.softmax_scale, A = (double)a.affine_a, Bc = (double)a.affine_b;
  kp.c_y = (float)(s * kLog2E / 36.0);
  const float c_a = (float)(A * s * kLog2E / 36.0);
  const float k0 = (float)(A * kLog2Of6 + Bc);
  kp.c_a8 = c_a * 0.125f;
  kp.k0_8 = k0 * 0.125f;
  kp.a8 = a.affine_a * 0.125f;
  kp.k1 = (float)kLog2Of6;
  kp.margin = (float)a.guard_margin;
  kp.floor_u = (float)(a.guard_shift + 1);
  kp.shift = (float)a.guard_shift;
  kp.out_bf16 = a.out_bf16;
  kp.row_ids = a.row_ids;
  kp.n_rows = a.n_rows;
  kp.p_codes = a.p_codes;
  kp.block_exp = a.block_exp;
  kp.row_m = a.row_m;
  kp.row_d = a.row_d;
  kp.wg_clock = a.wg_clock;
  kp.lse = a.lse;
  const bool dump = a.n_rows > 0;
  const int bh = a.B * a.H;
  // Eight waves (256 rows) per workgroup when that still fills the 256 CUs.
  // (the FP8 P/V route too: its d = 128 form spills a few registers with eight
  // waves, but four waves leave one per SIMD, since its LDS ring takes 108 KiB)
  // One exception: when the eight-wave grid takes two to five rounds and its last
  // round is at most half full, four-wave workgroups, two per CU, finish the tail
  // sooner (B1 N4096 d128: +9 % at H24, +10 % at H36, +4 % at H40, +3 % at H72;
  // -2 % with ten rounds at H64 N9472, and a full last round favours eight waves
  // by 4-7 %).  The FP8 route and the causal forward keep eight waves.
  // With d = 64 (FP4 P/V) the kernel runs at four waves per SIMD (one-step
  // pipeline; against three waves with two score buffers, +1-4 % on the paper's
  // D64 shapes, which in turn gained 7-10 % over two waves).  Eight-wave
  // workgroups, two per CU, when the eight-wave grid is a whole number of half
  // rounds (a multiple of 256 workgroups: +4-8 % at B1 N4096 H16-H128 and on the
  // paper's large shapes) and, for the causal forward, at least 3072 of them
  // (+2.5-5.7 %; -1 to -2 % at 1024-2048); otherwise four-wave workgroups, four
  // per CU (eight waves lost 6-15 % where the last half round is partly filled).
  const int64_t wide_wgs = a.N % 256 == 0 ? (int64_t)(a.N / 256) * bh : 0;
  const int64_t last_round = wide_wgs % 256;
  const bool tail = wide_wgs > 256 && wide_wgs <= 5 * 256 && last_round != 0 && last_round <= 128;
  const bool d64 = a.d == 64 && !a.pv_fp8;
  const bool d64_wide = wide_wgs >= 256 && last_round == 0 && (!a.causal || wide_wgs >= 3072);
  const bool wide = d64 ? d64_wide : (wide_wgs >= 256 && !(tail && !a.pv_fp8 && !a.causal));
  const int BM = wide ? 256 : 128;
  kp.n_qtiles = a.N / BM;
  kp.total = kp.n_qtiles * bh;
  const int ex2 = a.ex2_pairs;
  const int var = (a.guard ? kVarGuard : (a.causal ? kVarCausal : kVarOnline)) | (a.pv_fp8 ? kPV8 : 0);
  if (a.d == 128)
    return wide ? dispatch_dump<128, 8>(kp, dump, ex2, var, stream) : dispatch_dump<128, 4>(kp, dump, ex2, var, stream);
  return wide ? dispatch_dump<64, 8>(kp, dump, ex2, var, stream) : dispatch_dump<64, 4>(kp, dump, ex2, var, stream);
}

}  // namespace fp4attn
