// Direct-P full-MXFP4 attention forward for gfx950.
//
// Method (paper Sec. "Direct-P", Alg. 2, eqs. affine-code-map,
// represented-contributions, represented-output):
//   raw   = block-scaled FP4 product of Q and K          (= 36 Qhat Khat^T)
//   E_B   = floor(max_{j in B} raw_ij * c_y)              c_y = s log2(e) / 36
//   q_ij  = E2M1(max(0, fma(c_a, raw_ij, k0 - A E_B)))     c_a = A c_y, k0 = A log2 6 + B
//   O_i   = sum_B 2^(E_B - M_i) sum_j q_ij (6 Vhat_j) / (6 sum_B 2^(E_B - M_i) c_B)
//
// gfx950 design
// - One workgroup = NW waves = 32 * NW query rows of one (batch, head); each
//   wave owns 32 queries for the whole key loop.  Both products run on the
//   scaled FP4 matrix unit (v_mfma_scale_f32_32x32x64_f8f6f4) in transposed
//   form: S^T = K Q^T and O^T = V^T P^T.  Lane l then holds query l % 32 in
//   every accumulator, so the per-row online state (integer reference M_i, the
//   lazy power-of-two rescale) is a per-lane scalar and needs no cross-lane
//   broadcast.
// - Keys are fed to the S^T product in a permuted order (key_of_row below)
//   so that, with the 32x32 accumulator layout, lane half h holds all 32
//   scores of N32 block h of each 64-key step, in key order, in the registers
//   of two QK subtiles.  Block maximum, block exponent and E2M1 codes are then
//   lane-local, and the converted codes already form the lane's K64 P^T operand
//   of the PV product (the paper's two N32 fragments published as one K64
//   operand) with no cross-lane data movement.
// - Code map: one v_fma_f32 with the clamp modifier per score on u / 8 (the
//   median with 0 and 1 folds into it), then v_cvt_scalef32_pk_fp4_f32 with
//   scale 1/8 (two scores per instruction); the clamp realises max(0, u) and
//   saturation, and scaling by a power of two changes no rounding decision.
// - Native-exponential mixing (template EX2 = k of the 16 pairs of a block):
//   selected pairs take x = fma(c_y, raw, log2 6 - E_B) through v_exp_f32 and
//   the converter with scale 1, i.e. the ideal code Q_E2M1(2^x).
// - Causal variant: query i sees keys j <= i; a workgroup stops at the end of
//   its query tile, masked scores become -inf (code 0), and query tiles are
//   launched longest first.  Every variant can write the natural-log row
//   normaliser of the represented operator (LSE) for a backward pass.
// - Sampled guard (template VAR = kVarGuard, Alg. 3): the row reference is fixed from
//   the anchor keys of the first tile instead of following the block maxima;
//   working bytes are floored at L + 1 before the codes are formed and
//   published shifted down by L, so no rescale branch remains.
// - Denominator c_B: an extra 16x16x128 product of the same P^T register with a
//   constant indicator operand, so it uses exactly the codes and E8M0 bytes of
//   PV and costs no vector-ALU work.
// - K/V tiles of 128 keys are staged in LDS in matrix-operand order (each
//   lane's 16-byte fragment contiguous): a ring of four tiles filled three
//   tiles ahead by direct-to-LDS loads.  The key loop is software
//   pipelined two deep: while the vector ALU maps step g+1 to codes, the
//   matrix unit runs PV of step g and QK of step g+2.  With d = 64 and FP4 P/V
//   the loop runs one step deep at four waves per SIMD instead.
// - Workgroups are remapped so that the query tiles of one head run on one XCD
//   and share its L2 copy of that head's K/V.
#pragma once

#include <type_traits>

#include "gfx950.hpp"
#include "launch.hpp"

namespace fp4attn {
namespace directp_detail {

constexpr int kBN = 128;   // keys per LDS tile
constexpr int kTau = 32;   // lazy rescale: the reference may lag the row maximum by up to 32 binades
constexpr int kStages = 4; // LDS ring depth in tiles
// Row-reference variants of the kernel: the online integer reference, the
// sampled guard of Alg. 3, and the online reference with the causal mask;
// kPV8 added to a variant switches P and V to FP8 (E4M3) payloads.
constexpr int kVarOnline = 0, kVarGuard = 1, kVarCausal = 2, kPV8 = 8;
constexpr double kLog2E = 1.4426950408889634;
constexpr double kLog2Of6 = 2.584962500721156;

struct KParams {
  const uint8_t* qc;
  const uint8_t* qs;
  const uint8_t* kc;
  const uint8_t* ks;
  const uint8_t* vc;
  const uint8_t* vs;
  void* out;
  int N, n_qtiles, total;
  float c_y, c_a8, k0_8, a8, k1;
  float margin, floor_u, shift;  // sampled guard: M, L + 1, L
  int out_bf16;
  float* lse;  // optional [B, H, N] natural-log row normaliser
  const int64_t* row_ids;
  int n_rows;
  uint8_t* p_codes;
  int16_t* block_exp;
  int32_t* row_m;
  float* row_d;
  unsigned long long* wg_clock;
};

template <int D, bool PV8 = false>
struct Layout {
  static constexpr int kCodes = (kBN / 32) * (D / 64) * 1024;  // K fragments [sub][chunk][lane][16 B]
  static constexpr int kScales = (kBN / 32) * 64 * 4;          // [sub][lane] u32
  // V^T fragments [step][chunk][lane][16 B] (FP8: [step][chunk][half][lane][16 B],
  // the two 16-byte halves of a lane's 32-byte operand in separate planes, so
  // each read of a wave is one contiguous 1 KiB)
  static constexpr int vCodes = (kBN / 64) * (D / 32) * (PV8 ? 2048 : 1024);
  static constexpr int vScales = (D / 32) * 64 * 4;            // [chunk][lane] u32
  static constexpr int kOff = 0;
  static constexpr int ksOff = kOff + kCodes;
  static constexpr int vOff = ksOff + kScales;
  static constexpr int vsOff = vOff + vCodes;
  // E8M0 words as copied from global memory: the tile's K scales (contiguous,
  // d / 32 bytes per key), then one word of four 32-key block scales per V^T row
  static constexpr int rawK = kBN * (D / 32) / 4;  // words
  static constexpr int rawV = D;
  static constexpr int rawOff = vsOff + vScales;
  static constexpr int stage = rawOff + 4 * (rawK + rawV);
};

// Key order of the S^T product.  Operand row m = 8 g + 4 h + i of QK subtile
// `sub` (two subtiles per 64-key step) holds key 32 h + 16 (sub & 1) + 4 g + i of
// step sub / 2.  With the 32x32 accumulator layout, lane half h then holds all
// 32 keys of block h of the step, in key order, in the two subtiles' registers.
__device__ __forceinline__ int key_of_row(int sub, int m) {
  return 64 * (sub >> 1) + 32 * ((m >> 2) & 1) + 16 * (sub & 1) + 4 * (m >> 3) + (m & 3);
}
// Inverse: (subtile, operand row) of key k of a 128-key tile.
__device__ __forceinline__ int sub_of_key(int k) { return 2 * (k >> 6) + ((k >> 4) & 1); }
__device__ __forceinline__ int row_of_key(int k) { return 8 * ((k >> 2) & 3) + 4 * ((k >> 5) & 1) + (k & 3); }

// Direct-to-LDS buffer copies: lane l's 16 (4) bytes at byte soff + off of the
// buffer `rsrc` land at LDS byte address `lds` + 16 l (4 l); `lds` travels in
// M0, and one wait state separates its write from the load.  Bytes past the
// buffer's end read as zero, so a copy past the last tile is harmless.
// Written as inline assembly so that the compiler counts neither the loads
// nor the LDS they write (it would otherwise wait for every copy in flight
// before each LDS read); the kernel waits for its own copies with vm_wait
// before the barrier that publishes a tile.
// (`lds` and `soff` are wave-uniform; reading them from the first lane keeps
// them in scalar registers whatever the compiler's uniformity analysis says.)
__device__ __forceinline__ void lds_copy16(unsigned lds, __amdgpu_buffer_rsrc_t rsrc, int soff, unsigned off) {
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(off), "s"(rsrc),
               "s"(__builtin_amdgcn_readfirstlane(soff)), "{m0}"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}
__device__ __forceinline__ void lds_copy4(unsigned lds, __amdgpu_buffer_rsrc_t rsrc, int soff, unsigned off) {
  asm volatile("s_nop 0\n\tbuffer_load_dword %0, %1, %2 offen lds" ::"v"(off), "s"(rsrc),
               "s"(__builtin_amdgcn_readfirstlane(soff)), "{m0}"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}
// Wait until at most n of this wave's vector-memory operations are in flight.
template <int n>
__device__ __forceinline__ void vm_wait() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n) : "memory");
}
__device__ __forceinline__ unsigned lds_address(const uint8_t* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
}
// Raw buffer over `bytes` bytes (gfx9 descriptor: 32-bit data format, no stride).
// Base and size are the same in every lane; reading them from the first lane
// keeps the descriptor in scalar registers, as the copy instructions require.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_buffer(const uint8_t* base, int bytes) {
  const uint64_t a = (uint64_t)base;
  const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)a), hi = __builtin_amdgcn_readfirstlane((unsigned)(a >> 32));
  uint8_t* b = (uint8_t*)(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(b, (short)0, __builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

// One 128-key tile: K and V^T codes copied from global memory straight into an
// LDS stage in operand order, and its E8M0 words copied raw, then rearranged
// in LDS by the wave that copied them.
//   Codes: item i is one 16-byte operand fragment, K items first, then V^T
//   items; thread tid copies items tid, tid + NT, ...  A wave's 64 lanes copy
//   64 consecutive fragments, the order in which the direct-to-LDS load writes.
//   Scales: 64 raw words per block; wave w copies block w % kRawWaves, so
//   with more waves than blocks two waves write the same bytes to the same
//   place, and every wave issues the same number of loads per tile.
// A copy reads one buffer of the (batch, head) at this lane's fixed offset
// plus a per-tile scalar offset (key0 / 2) * mul (scales: (key0 / 32) * mul);
// the buffer, the multiplier and the LDS position are fixed per wave.
template <int D, int NW, bool PV8>
struct TileCopy {
  using L = Layout<D, PV8>;
  static constexpr int NT = NW * 64;
  static constexpr int nK = L::kCodes / 16;
  static constexpr int nV = L::vCodes / 16;
  static constexpr int kItems = nK + nV;
  static constexpr int kPerThread = (kItems + NT - 1) / NT;
  static constexpr int kRawWaves = (L::rawK + L::rawV) / 64;  // blocks of 64 raw words
  static constexpr int kLoads = kItems / NT + 1;              // loads every wave issues per tile, at least
  static_assert(nK % 64 == 0 && nV % 64 == 0, "whole waves per operand");
  static_assert(L::rawK % 64 == 0 && L::rawV % 64 == 0 && kRawWaves <= NW, "whole waves per scale operand");

  __amdgpu_buffer_rsrc_t buf[kPerThread], raw_buf;  // wave-uniform
  int mul[kPerThread], raw_mul;                     // wave-uniform
  unsigned lds_off[kPerThread], raw_lds;            // wave-uniform
  unsigned off[kPerThread], raw_off;                // this lane's offsets
  bool active[kPerThread];                          // wave-uniform

  __device__ __forceinline__ void init(const uint8_t* kc, const uint8_t* ks, const uint8_t* vc, const uint8_t* vs,
                                       int N, int tid) {
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const __amdgpu_buffer_rsrc_t kbuf = make_buffer(kc, N * (D / 2));
    const __amdgpu_buffer_rsrc_t vbuf = make_buffer(vc, D * (PV8 ? N : N / 2));
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int item0 = wave * 64 + i * NT, item = item0 + lane;
      active[i] = kItems % NT == 0 || item0 < kItems;
      const bool is_k = (nK % NT == 0) ? (i < nK / NT) : item0 < nK;  // compile-time where it can be
      buf[i] = is_k ? kbuf : vbuf;
      mul[i] = is_k ? D : (PV8 ? 2 : 1);
      lds_off[i] = is_k ? L::kOff + item0 * 16 : L::vOff + (item0 - nK) * 16;
      if (is_k) {
        const int m = item & 63, rest = item >> 6;
        const int c = rest % (D / 64), sub = rest / (D / 64);
        off[i] = key_of_row(sub, m & 31) * (D / 2) + (2 * c + (m >> 5)) * 16;
      } else if constexpr (PV8) {
        // One byte per key.  The FP8 operand's k order: lane half h holds keys
        // 16 h + [0, 16) (bytes 0-15) and 32 + 16 h + [0, 16) (bytes 16-31) of
        // the 64-key step, while its E8M0 byte still covers keys 32 h + [0, 32).
        const int vi = item - nK;
        const int m = vi & 63, hh = (vi >> 6) & 1, rest = vi >> 7;
        const int cc = rest % (D / 32), s = rest / (D / 32);
        off[i] = (cc * 32 + (m & 31)) * N + s * 64 + (m >> 5) * 16 + hh * 32;
      } else {
        const int vi = item - nK;
        const int m = vi & 63, rest = vi >> 6;
        const int cc = rest % (D / 32), s = rest / (D / 32);
        off[i] = (cc * 32 + (m & 31)) * (N / 2) + s * 32 + (m >> 5) * 16;
      }
    }
    const int rb = wave % kRawWaves, r = rb * 64 + lane;
    const bool raw_k = rb * 64 < L::rawK;
    raw_buf = raw_k ? make_buffer(ks, N * (D / 32)) : make_buffer(vs, D * (N / 32));
    raw_mul = raw_k ? D : 1;  // per 32 keys: d / 32 bytes for each of 32 keys, or one byte
    raw_lds = L::rawOff + rb * 256;
    raw_off = raw_k ? 4 * r : (r - L::rawK) * (N / 32);
  }

  // Fetch the tile of keys [key0, key0 + 128) into stage `st`.
  __device__ __forceinline__ void issue(uint8_t* st, int key0) const {
    const unsigned lds = lds_address(st);
    const int half = key0 >> 1;
#pragma unroll
    for (int i = 0; i < kPerThread; ++i)
      if (active[i]) lds_copy16(lds + lds_off[i], buf[i], half * mul[i], off[i]);
    lds_copy4(lds + raw_lds, raw_buf, (key0 >> 5) * raw_mul, raw_off);
  }

  // The tile's E8M0 words in operand order: K word of key k at [sub][row] and,
  // shifted by one byte, at [sub][row + 32] (lanes 0..31 take scale bytes 0 and 2
  // of a word, lanes 32..63 bytes 1 and 3); V^T words likewise per 32-row chunk.
  // Reads only raw words this wave copied itself.
  __device__ __forceinline__ static void arrange(uint8_t* st, int tid) {
    const int wave = tid >> 6, r = tid;  // wave w < kRawWaves arranges block w
    if (wave >= kRawWaves) return;
    const unsigned raw = reinterpret_cast<const uint32_t*>(st + L::rawOff)[r];
    auto put_k = [&](int key, unsigned w) {
      uint32_t* dst = reinterpret_cast<uint32_t*>(st + L::ksOff) + sub_of_key(key) * 64 + row_of_key(key);
      dst[0] = w;
      dst[32] = w >> 8;
    };
    if (r < L::rawK) {
      if constexpr (D == 128) {
        put_k(r, raw);
      } else {  // two keys of two bytes
        put_k(2 * r, raw & 0xffff);
        put_k(2 * r + 1, raw >> 16);
      }
    } else {
      const int row = r - L::rawK;
      uint32_t* dst = reinterpret_cast<uint32_t*>(st + L::vsOff) + (row >> 5) * 64 + (row & 31);
      dst[0] = raw;
      dst[32] = raw >> 8;
    }
  }
};

// The FP4 P/V routes with d = 64 pipeline the key loop one step deep (one S^T
// buffer, one P operand) to fit 128 registers: four waves per SIMD, i.e. four
// four-wave or two eight-wave workgroups of 40 KiB LDS per CU.
template <int D, int NW, int VAR>
constexpr bool kOneBuffer = D == 64 && (VAR & kPV8) == 0;
// Two waves per SIMD, except where the LDS ring allows one workgroup of four
// waves per CU only (FP8 V tiles with d = 128: 108 KiB), and four for the
// one-buffer form above.
template <int D, int NW, int VAR>
constexpr int kMinWaves = (VAR & kPV8) ? ((NW == 4 && D == 128) ? 1 : 2)
                                       : (kOneBuffer<D, NW, VAR> ? 4 : ((D == 64 && NW == 4) ? 3 : 2));
template <int D, int NW, int VAR>
constexpr int kMaxWaves = kMinWaves<D, NW, VAR> > 2 ? kMinWaves<D, NW, VAR> : 2;

template <int D, int NW, bool DUMP, int EX2, int VAR>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(kMinWaves<D, NW, VAR>, kMaxWaves<D, NW, VAR>))) void
fwd_mxfp4_kernel(const KParams p) {
  constexpr bool PV8 = (VAR & kPV8) != 0;  // FP8 (E4M3) P and V payloads
  constexpr bool GUARD = (VAR & 7) == kVarGuard, CAUSAL = (VAR & 7) == kVarCausal;
  static_assert(!(PV8 && (GUARD || EX2 != 0)), "the FP8 route takes the exponential on every key");
  using POp = std::conditional_t<PV8, v8i, v4i>;  // a lane's 32 P payloads
  static_assert(EX2 == 0 || EX2 == 1 || EX2 == 2 || EX2 == 4 || EX2 == 8 || EX2 == 16, "pairs per 32-key block");
  using L = Layout<D, (VAR & kPV8) != 0>;
  constexpr int BM = NW * 32;
  // The LDS ring: one array per stage, so that the compiler tracks the
  // direct-to-LDS copies per stage and waits for none of them before reading
  // another stage.
  __shared__ __attribute__((aligned(16))) uint8_t ring0[L::stage];
  __shared__ __attribute__((aligned(16))) uint8_t ring1[L::stage];
  __shared__ __attribute__((aligned(16))) uint8_t ring2[L::stage];
  __shared__ __attribute__((aligned(16))) uint8_t ring3[L::stage];
  static_assert(kStages == 4, "one array per ring stage");
  auto ring = [&](auto B_) -> uint8_t* {
    constexpr int b = decltype(B_)::value % kStages;
    if constexpr (b == 0) return ring0;
    else if constexpr (b == 1) return ring1;
    else if constexpr (b == 2) return ring2;
    else return ring3;
  };
  using I0 = std::integral_constant<int, 0>;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, h = lane >> 5, lr = lane & 31;
  const unsigned long long clk0 = __builtin_amdgcn_s_memtime(), rt0 = __builtin_amdgcn_s_memrealtime();
  int bh, qt;
  if constexpr (CAUSAL) {
    // longest query tiles first, spread over the XCDs in launch order
    const int n_bh = p.total / p.n_qtiles;
    bh = blockIdx.x % n_bh;
    qt = p.n_qtiles - 1 - blockIdx.x / n_bh;
  } else {
    const int lin = xcd_remap(blockIdx.x, p.total);
    bh = lin / p.n_qtiles;
    qt = lin % p.n_qtiles;
  }
  const int N = p.N;
  const int qrow = qt * BM + wave * 32 + lr;

  const uint8_t* kc = p.kc + (size_t)bh * N * (D / 2);
  const uint8_t* ks = p.ks + (size_t)bh * N * (D / 32);
  const uint8_t* vc = p.vc + (size_t)bh * D * (PV8 ? N : N / 2);
  const uint8_t* vs = p.vs + (size_t)bh * D * (N / 32);

  // Q^T operand, resident for the whole key loop.
  v4i qf[D / 64];
  {
    const uint8_t* qrow_codes = p.qc + ((size_t)bh * N + qrow) * (D / 2);
#pragma unroll
    for (int c = 0; c < D / 64; ++c) qf[c] = *reinterpret_cast<const v4i*>(qrow_codes + (2 * c + h) * 16);
  }
  int qsc;
  {
    const uint8_t* qs = p.qs + ((size_t)bh * N + qrow) * (D / 32);
    const unsigned raw = D == 128 ? *reinterpret_cast<const uint32_t*>(qs) : *reinterpret_cast<const uint16_t*>(qs);
    qsc = (int)(raw >> (8 * h));
  }

  int slot = -1;
  if constexpr (DUMP) {
    const int64_t g = (int64_t)bh * N + qrow;
    int lo = 0, hi = p.n_rows - 1;
    while (lo <= hi) {
      const int mid = (lo + hi) >> 1;
      const int64_t v = p.row_ids[mid];
      if (v == g) {
        slot = mid;
        break;
      }
      if (v < g) lo = mid + 1;
      else hi = mid - 1;
    }
  }

  // Denominator operand.  Read as the B operand of a 16x16x128 product, the K64
  // P^T register of lane l is column l % 16 and K-block l / 16, i.e. query
  // (l % 32)'s keys 32 (l / 32) .. +31.  Row 0 of this indicator matrix selects
  // K-blocks 0 and 2 (query c's 64 keys), row 1 K-blocks 1 and 3 (query c + 16),
  // so one 16x16x128 product yields every query's code sum with the P scales.
  // FP8: the 16x16x128 form's K-blocks mix queries c and c + 16 under one
  // scale, so the FP8 denominator is row 0 of a 32x32x64 product instead, whose
  // indicator row 0 (lanes 0 and 32) is all ones.
  const bool one_lane = PV8 ? (lane == 0 || lane == 32) : (lane == 0 || lane == 32 || lane == 17 || lane == 49);
  const int ones_word = one_lane ? (PV8 ? 0x38383838 : 0x22222222) : 0;  // E4M3 / E2M1 1.0
  POp ones;
#pragma unroll
  for (int i = 0; i < (PV8 ? 8 : 4); ++i) ones[i] = ones_word;

  v16f O[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c) O[c] = v16f{};
  // FP4: lane c < 16, register 0 = query c, register 1 = query c + 16.
  // FP8: lane c < 32, register 0 = query c.
  std::conditional_t<PV8, v16f, v4f> Dacc = {};
  float Mref = -1.0e6f;  // integer row reference (exact in fp32); no block seen yet
  // Carried with it: the rescale threshold M + tau and the E8M0 bias, so that a
  // block's byte is one subtraction from E (all small integers, exact in fp32).
  constexpr float kByteBias = PV8 ? 120.0f : 127.0f;
  float Mthr = Mref + kTau, Mbias = Mref - kByteBias;
  // -A / 8 held in a vector register: the code-map offset fma then reads one
  // scalar operand only and needs no per-step copy (emits nothing).
  float na8 = -p.a8;
  asm volatile("" : "+v"(na8));
  float Rref = 0.0f;     // guard: fixed row reference from the anchor tile (Alg. 3)

  const int ntiles = CAUSAL ? (qt + 1) * BM / kBN : N / kBN;  // causal: keys up to the tile's last query
  const int nsteps = 2 * ntiles;  // 64-key steps

  // S^T of 64-key step `sl` (0 or 1) of the tile held in `st`: two 32-key blocks.
  auto qk = [&](const uint8_t* st, auto SL_, v16f(&acc)[2]) {
    constexpr int sl = decltype(SL_)::value;
    static_for<2>([&](auto T_) {
      constexpr int t = decltype(T_)::value;
      constexpr int sub = 2 * sl + t;
      v16f a = v16f{};
      const int ksc = reinterpret_cast<const int*>(st + L::ksOff)[sub * 64 + lane];
      static_for<D / 64>([&](auto C_) {
        constexpr int c = decltype(C_)::value;
        const v4i kf = *reinterpret_cast<const v4i*>(st + L::kOff + ((sub * (D / 64) + c) * 64 + lane) * 16);
        a = mfma_fp4_32x32x64<2 * c, 2 * c>(kf, qf[c], a, ksc, qsc);
      });
      acc[t] = a;
    });
  };

  // PV of step `s` (0 or 1) of the tile held in `st`, and the represented
  // denominator from the same P^T operand and E8M0 bytes.
  auto pv = [&](const uint8_t* st, auto S_, const POp& P, int u) {
    constexpr int s = decltype(S_)::value;
    static_for<D / 32>([&](auto C_) {
      constexpr int c = decltype(C_)::value;
      const int vsc = reinterpret_cast<const int*>(st + L::vsOff)[c * 64 + lane];
      if constexpr (PV8) {
        const uint8_t* vp = st + L::vOff + (s * (D / 32) + c) * 2048 + lane * 16;
        const v4i v0 = *reinterpret_cast<const v4i*>(vp), v1 = *reinterpret_cast<const v4i*>(vp + 1024);
        const v8i vf = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
        O[c] = mfma_fp8_32x32x64<2 * s, 0>(vf, P, O[c], vsc, u);
      } else {
        const v4i vf = *reinterpret_cast<const v4i*>(st + L::vOff + ((s * (D / 32) + c) * 64 + lane) * 16);
        O[c] = mfma_fp4_32x32x64<2 * s, 0>(vf, P, O[c], vsc, u);
      }
    });
    if constexpr (PV8) Dacc = mfma_fp8_32x32x64<0, 0>(ones, P, Dacc, 127, u);
    else Dacc = mfma_fp4_16x16x128<0, 0>(ones, P, Dacc, 127, u);
  };

  // Instruction order of one steady-state step (the region before the rescale
  // branch): the step's LDS operand reads first, the block-maximum chain while
  // they land, then every MFMA followed by a slice of the code map.
  auto schedule_step = [&]() {
    __builtin_amdgcn_sched_group_barrier(0x100, 12, 0);  // DS reads: V, K fragments and scales
    __builtin_amdgcn_sched_group_barrier(0x002, 18, 0);  // VALU: block maximum, exponent, offset
    static_for<D / 32 + 1 + 2 * (D / 64)>([&](auto) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);  // six VALU of the code map
    });
  };

  // Direct-P for global 64-key step g (Alg. 2, steps 1-6).  Lane half h holds
  // the 32 scores of block h of the step for query l % 32 (acc[0]: keys 0-15,
  // acc[1]: keys 16-31), so the block maximum, the block exponent and the codes
  // are all lane-local, and the codes land in the K64 P^T operand as they are
  // converted.  Only the rare rescale branch exchanges the two halves' exponents.
  auto directp = [&](const v16f(&acc)[2], int g, POp& P, int& u, auto SCHED_) {
    // 32 values in 16 three-input maxima (v_max3_f32)
    float m = fmaxf(fmaxf(acc[0][0], acc[0][1]), acc[0][2]);
#pragma unroll
    for (int r = 3; r < 15; r += 2) m = fmaxf(fmaxf(m, acc[0][r]), acc[0][r + 1]);
    m = fmaxf(fmaxf(m, acc[0][15]), acc[1][0]);
#pragma unroll
    for (int r = 1; r < 15; r += 2) m = fmaxf(fmaxf(m, acc[1][r]), acc[1][r + 1]);
    m = fmaxf(m, acc[1][15]);
    // Block exponent (Alg. 2, step 2) and the offset T of the code map,
    // x = y - T + log2 6.  Online reference: T = E_B = floor(max y).  Guard
    // (Alg. 3, step 3): e_B = floor(max y - R), working byte ubar_B =
    // clamp(e_B + 127, L + 1, 254), T = R + ubar_B - 127 (every step rounded
    // to fp32 on its own).
    float E, T, ub = 0.0f;
    if constexpr (GUARD) {
#pragma clang fp contract(off)
      const float Y = m * p.c_y;
      ub = __builtin_amdgcn_fmed3f(floorf(Y - Rref) + 127.0f, p.floor_u, 254.0f);
      E = ub - 127.0f;
      T = Rref + E;
    } else {
      E = floorf(m * p.c_y);
      // causal: a block with no visible key has E = -inf; a finite offset keeps
      // its codes at 0 instead of NaN (its E8M0 byte is 0 either way)
      T = CAUSAL ? fmaxf(E, -1.0e30f) : E;
    }
    const float c0 = fmaf(na8, T, p.k0_8);      // (A (log2 6 - T) + B) / 8
    const float c1 = EX2 ? p.k1 - T : 0.0f;     // log2 6 - T, the exponent offset of 2^x
    if constexpr (PV8) {
      // FP8 payload: E4M3(2^(y - T + 7)) < 256 for every key (the block maximum
      // in [128, 256)); word w holds keys 4 w .. 4 w + 3.
      const float c7 = 7.0f - T;
      unsigned w8[8];  // key order: words 0-3 keys 0-15 of the lane's block, 4-7 keys 16-31
      static_for<8>([&](auto W_) {
        constexpr int w = decltype(W_)::value;
        constexpr int r0 = 4 * (w % 4);
        const float e0 = __builtin_amdgcn_exp2f(fmaf(p.c_y, acc[w / 4][r0], c7));
        const float e1 = __builtin_amdgcn_exp2f(fmaf(p.c_y, acc[w / 4][r0 + 1], c7));
        const float e2 = __builtin_amdgcn_exp2f(fmaf(p.c_y, acc[w / 4][r0 + 2], c7));
        const float e3 = __builtin_amdgcn_exp2f(fmaf(p.c_y, acc[w / 4][r0 + 3], c7));
        w8[w] = cvt_pk_fp8<true>(cvt_pk_fp8<false>(as_uint(e0), e0, e1), e2, e3);
      });
      if constexpr (DUMP) {
        if (slot >= 0) {
          const v8i keyorder = {(int)w8[0], (int)w8[1], (int)w8[2], (int)w8[3],
                                (int)w8[4], (int)w8[5], (int)w8[6], (int)w8[7]};
          *reinterpret_cast<v8i*>(p.p_codes + (size_t)slot * N + (2 * g + h) * 32) = keyorder;
        }
      }
      // Operand k order (see TileCopy::issue): the lower half keeps keys 0-15 of
      // block 0 and takes keys 0-15 of block 1; the upper half takes keys 16-31
      // of block 0 and keeps keys 16-31 of block 1.
#pragma unroll
      for (int i = 0; i < 4; ++i) swap_halves(w8[i], w8[i + 4]);
#pragma unroll
      for (int i = 0; i < 8; ++i) P[i] = (int)w8[i];
    } else {
      // Code map on u / 8.  Every byte of the four words is written below; the
      // first convert of each word takes its own input as the overwritten value.
      unsigned w[4];
      static_for<4>([&](auto I_) {
        constexpr int i = decltype(I_)::value;
        static_for<4>([&](auto W_) {
          constexpr int wd = decltype(W_)::value;  // word wd holds keys 8 wd .. 8 wd + 7
          const float s_lo = acc[wd / 2][8 * (wd % 2) + 2 * i], s_hi = acc[wd / 2][8 * (wd % 2) + 2 * i + 1];
          // pair 4 wd + i of the block (keys 8 wd + 2 i and 8 wd + 2 i + 1)
          if constexpr (EX2 != 0 && (4 * wd + i) % (16 / (EX2 ? EX2 : 1)) == 0) {
            const float lo = __builtin_amdgcn_exp2f(fmaf(p.c_y, s_lo, c1));
            const float hi = __builtin_amdgcn_exp2f(fmaf(p.c_y, s_hi, c1));
            w[wd] = cvt_pk_fp4<i>(i == 0 ? as_uint(lo) : w[wd], lo, hi, 1.0f);
          } else {
            const float lo = __builtin_amdgcn_fmed3f(fmaf(p.c_a8, s_lo, c0), 0.0f, 1.0f);
            const float hi = __builtin_amdgcn_fmed3f(fmaf(p.c_a8, s_hi, c0), 0.0f, 1.0f);
            w[wd] = cvt_pk_fp4<i>(i == 0 ? as_uint(lo) : w[wd], lo, hi, 0.125f);
          }
        });
      });
      P = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
    }
    // Keep the code map in this basic block, next to the step's matrix work,
    // instead of letting it sink below the rescale branch (emits nothing).
    if constexpr (PV8) {
      // (a 256-bit operand would not pass the host compiler's asm checks)
      const v4i p_lo = __builtin_shufflevector(P, P, 0, 1, 2, 3), p_hi = __builtin_shufflevector(P, P, 4, 5, 6, 7);
      asm volatile("" ::"v"(p_lo), "v"(p_hi));
    } else {
      asm volatile("" ::"v"(P));
    }
    if constexpr (decltype(SCHED_)::value) schedule_step();
    if constexpr (GUARD) {
      // published byte ubar_B - L, in [1, 254 - L]
      u = (int)__builtin_amdgcn_cvt_pk_u8_f32(ub - p.shift, 0, 0u);
      // The rescale branch of the online reference is where the accumulators
      // pass between steps; without it the compiler regroups the PV chains of
      // several steps and runs out of registers.  Pass them through here
      // (emits nothing).
#pragma unroll
      for (int c = 0; c < D / 32; ++c) asm volatile("" : "+v"(O[c]));
      asm volatile("" : "+v"(Dacc));
    } else {
      // Online integer reference with a lazy, exact power-of-two rescale of what
      // PV has accumulated so far; the halves agree on the reference because the
      // branch is taken by the whole wave and uses both halves' exponents.
      if (__builtin_amdgcn_ballot_w64(E > Mthr)) {
        unsigned ea = as_uint(E), eb = ea;
        swap_halves(ea, eb);  // each lane: (block-0 exponent, block-1 exponent)
        const float Emax = fmaxf(as_float(ea), as_float(eb));
        const float Mn = Emax > Mthr ? Emax : Mref;
        const int sh = (int)(Mref - Mn);
#pragma unroll
        for (int c = 0; c < D / 32; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) O[c][r] = ldexpf(O[c][r], sh);
        Dacc[0] = ldexpf(Dacc[0], sh);
        if constexpr (!PV8) Dacc[1] = ldexpf(Dacc[1], lane_read(sh, (lane + 16) & 63));  // query lane + 16
        Mref = Mn;
        Mthr = Mn + kTau;
        Mbias = Mn - kByteBias;
      }
      // E8M0 byte of this lane's block: clamp(E - M + 127, 0, 254) (E - M <= kTau).
      u = (int)__builtin_amdgcn_cvt_pk_u8_f32(E - Mbias, 0, 0u);
    }
    if constexpr (DUMP) {
      if (slot >= 0) {
        const int kb = 2 * g + h;
        if constexpr (!PV8) *reinterpret_cast<v4i*>(p.p_codes + (size_t)slot * (N / 2) + kb * 16) = P;
        // -32768 marks a block with no visible key (causal mask)
        p.block_exp[(size_t)slot * (N / 32) + kb] = (int16_t)(E > -32768.0f ? (int)E : -32768);
      }
    }
  };

  // Causal mask of 64-key step g: lane half h holds keys 64 g + 32 h + 16 t + r
  // (register r of subtile t) for query qrow; keys after the query become -inf.
  // Only steps that reach past the wave's first query need it (wave-uniform).
  auto causal_mask = [&](v16f(&acc)[2], int g) {
    if (64 * g + 63 > qt * BM + wave * 32) {
      const int lim = qrow - (64 * g + 32 * h);  // last visible offset in this lane's block
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (16 * t + r > lim) acc[t][r] = -__builtin_inff();
    }
  };

  // Pipeline.  LDS holds a ring of kStages = 4 tiles.  At the start of tile t
  // each wave waits until its copies of tile t+1 have landed (only tile t+2's
  // may still be in flight), puts the E8M0 words it copied into operand order,
  // and after the barrier fetches tile t+3 into the stage of tile t-1, which
  // every wave has finished reading.  Every publish fetches exactly one tile
  // (past the end: bounds-checked bytes, zero past each buffer's end, into a
  // stage nobody reads), so a wave's vmcnt always counts the same loads.  In 64-key step g the matrix unit runs
  // PV of step g and QK of step g+2 while the vector ALU runs Direct-P of step
  // g+1.  Steps are unrolled eight at a time (four tiles), so every LDS stage is
  // a compile-time constant.
  using Copy = TileCopy<D, NW, PV8>;
  constexpr int kBatch = Copy::kLoads;
  Copy copy;
  copy.init(kc, ks, vc, vs, N, tid);
  copy.issue(ring(I0{}), 0);
  copy.issue(ring(std::integral_constant<int, 1>{}), kBN);
  copy.issue(ring(std::integral_constant<int, 2>{}), 2 * kBN);
  vm_wait<2 * kBatch>();  // tile 0 has landed
  Copy::arrange(ring(I0{}), tid);
  __syncthreads();

  if constexpr (kOneBuffer<D, NW, VAR>) {
    // One step deep: step g runs PV(g), then QK(g+1) and its code map, which
    // waits for those products; the other waves of the SIMD fill the wait.  The
    // tile that QK(g+1) reads first is published in the step before it (the
    // second step of a tile), by the same waits, barrier and copy as below.
    v16f S1[2];
    POp P1;
    int u1;
    if constexpr (GUARD) {
      // Anchor (Alg. 3, steps 1-2) over both steps of the first key tile, one step
      // at a time; the buffer ends with step 0's scores for its code map.
      float am = -__builtin_inff();
      static_for<2>([&](auto T_) {
        qk(ring(I0{}), std::integral_constant<int, 1 - decltype(T_)::value>{}, S1);
#pragma unroll
        for (int r = 0; r < 16; ++r) am = fmaxf(fmaxf(am, S1[0][r]), S1[1][r]);
      });
      unsigned ma = as_uint(am), mb = ma;
      swap_halves(ma, mb);
      {
#pragma clang fp contract(off)
        const float Y = fmaxf(as_float(ma), as_float(mb)) * p.c_y;
        Rref = Y + p.margin;
      }
    } else {
      qk(ring(I0{}), std::integral_constant<int, 0>{}, S1);
    }
    if constexpr (CAUSAL) causal_mask(S1, 0);
    directp(S1, 0, P1, u1, std::false_type{});
    auto step1 = [&](auto J_, auto TAIL_, int g) {
      constexpr int j = decltype(J_)::value;
      constexpr bool guard = decltype(TAIL_)::value;
      constexpr int sl = j % 2;
      using b_cur = std::integral_constant<int, j / 2>;
      using b_nxt = std::integral_constant<int, j / 2 + 1>;
      using b_new = std::integral_constant<int, j / 2 + 3>;
      const int t = g >> 1;
      pv(ring(b_cur{}), std::integral_constant<int, sl>{}, P1, u1);
      if constexpr (sl == 1) {
        vm_wait<kBatch>();  // tile t+1 has landed: only tile t+2's loads may be in flight
        if (!guard || t + 1 < ntiles) Copy::arrange(ring(b_nxt{}), tid);
        __syncthreads();
        copy.issue(ring(b_new{}), (t + 3) * kBN);
      }
      if (!guard || g + 1 < nsteps) {
        if constexpr (sl == 0) qk(ring(b_cur{}), std::integral_constant<int, 1>{}, S1);
        else qk(ring(b_nxt{}), std::integral_constant<int, 0>{}, S1);
        // masked steps all fall in the tail group (see the loop bound below)
        if constexpr (CAUSAL && guard) causal_mask(S1, g + 1);
        directp(S1, g + 1, P1, u1, std::false_type{});
      }
    };
    // As below: the tail group holds every step whose keys reach past a query of
    // the tile (Direct-P of step g' >= nsteps - BM / 64 runs in step g' - 1).
    constexpr int kLeft1 = CAUSAL ? BM / 64 + 1 : 2;
    int g0 = 0;
    for (; g0 + 8 <= nsteps - kLeft1; g0 += 8) {
      static_for<8>([&](auto J_) { step1(J_, std::false_type{}, g0 + decltype(J_)::value); });
    }
    static_for<8 + kLeft1>([&](auto J_) {  // tail: fewer than 8 + kLeft1 steps remain
      const int g = g0 + decltype(J_)::value;
      if (g < nsteps) step1(J_, std::true_type{}, g);
    });
  } else {
    // Two S^T buffers and two P operands alternate with the step parity.
    v16f SA[2], SB[2];
    POp PA, PB;
    int uA, uB;
    if constexpr (GUARD) {
      // Anchor (Alg. 3, steps 1-2): the largest score of the first key tile, which
      // holds the anchor keys; each lane half has two of its four 32-key blocks.
      qk(ring(I0{}), std::integral_constant<int, 0>{}, SB);
      qk(ring(I0{}), std::integral_constant<int, 1>{}, SA);
      float am = fmaxf(SB[0][0], SB[1][0]);
#pragma unroll
      for (int r = 0; r < 16; ++r) am = fmaxf(fmaxf(am, SB[0][r]), SB[1][r]);
#pragma unroll
      for (int r = 0; r < 16; ++r) am = fmaxf(fmaxf(am, SA[0][r]), SA[1][r]);
      unsigned ma = as_uint(am), mb = ma;
      swap_halves(ma, mb);
      {
#pragma clang fp contract(off)
        const float Y = fmaxf(as_float(ma), as_float(mb)) * p.c_y;
        Rref = Y + p.margin;
      }
      directp(SB, 0, PA, uA, std::false_type{});
    } else {
      qk(ring(I0{}), std::integral_constant<int, 0>{}, SA);
      if constexpr (CAUSAL) causal_mask(SA, 0);
      directp(SA, 0, PA, uA, std::false_type{});
      qk(ring(I0{}), std::integral_constant<int, 1>{}, SA);
    }

    // One step of the pipeline; j is the step's position in its group of eight.
    // TAIL: the tail group, where QK, Direct-P or the step itself may not exist.
    auto step = [&](auto J_, auto TAIL_, int g) {
      constexpr int j = decltype(J_)::value;
      constexpr bool guard = decltype(TAIL_)::value;
      constexpr int sl = j % 2;                 // step within its tile
      using b_cur = std::integral_constant<int, j / 2>;  // ring stage of tile t
      using b_nxt = std::integral_constant<int, j / 2 + 1>;
      using b_new = std::integral_constant<int, j / 2 + 3>;
      auto& S_in = (sl == 0) ? SA : SB;   // S^T of step g+1
      auto& S_out = (sl == 0) ? SB : SA;  // S^T of step g+2
      auto& P_cur = (sl == 0) ? PA : PB;  // P of step g
      auto& u_cur = (sl == 0) ? uA : uB;
      auto& P_nxt = (sl == 0) ? PB : PA;  // P of step g+1
      auto& u_nxt = (sl == 0) ? uB : uA;
      const int t = g >> 1;
      // PV of step g and Direct-P of step g+1 read nothing the barrier publishes,
      // so they come first: the matrix unit has PV's products in hand while the
      // waves meet at the barrier.
      pv(ring(b_cur{}), std::integral_constant<int, sl>{}, P_cur, u_cur);
      if (!guard || g + 1 < nsteps) {
        // masked steps all fall in the tail group (see the loop bound below)
        if constexpr (CAUSAL && guard) causal_mask(S_in, g + 1);
        directp(S_in, g + 1, P_nxt, u_nxt, std::bool_constant<!guard>{});
      }
      if constexpr (sl == 0) {
        vm_wait<kBatch>();  // tile t+1 has landed: only tile t+2's loads may be in flight
        if (!guard || t + 1 < ntiles) Copy::arrange(ring(b_nxt{}), tid);
        __syncthreads();
        copy.issue(ring(b_new{}), (t + 3) * kBN);
      }
      if (!guard || g + 2 < nsteps) {
        qk(ring(b_nxt{}), std::integral_constant<int, sl>{}, S_out);
        // Issue QK of step g+2 in this step (it would otherwise sink next to its
        // consumer in step g+1 and serialise with the code map); emits nothing.
        asm volatile("" ::"v"(S_out[0]), "v"(S_out[1]));
      }
    };


    // The unrolled loop stops kLeft steps before the end, so that the tail group
    // holds every step that may lack QK or Direct-P work and, with the causal
    // mask, every step whose keys reach past a query of the tile: Direct-P of
    // step g' >= nsteps - BM / 64 runs in step g' - 1.
    constexpr int kLeft = CAUSAL ? BM / 64 + 1 : 2;
    int g0 = 0;
    for (; g0 + 8 <= nsteps - kLeft; g0 += 8) {
      static_for<8>([&](auto J_) { step(J_, std::false_type{}, g0 + decltype(J_)::value); });
    }
    // tail: fewer than 8 + kLeft steps remain
    static_for<8 + kLeft>([&](auto J_) {
      const int g = g0 + decltype(J_)::value;
      if (g < nsteps) step(J_, std::true_type{}, g);
    });
  }
  vm_wait<0>();  // no copy may still be landing in LDS when the workgroup ends

  // Epilogue: O = acc / (6 D).  The denominator sits in register 0 of the lower half.
  float Dfin;  // query lane % 32
  if constexpr (PV8) {
    Dfin = lane_read(Dacc[0], lane & 31);
  } else {
    const float d_lo = lane_read(Dacc[0], lane & 15), d_hi = lane_read(Dacc[1], lane & 15);
    Dfin = (lane & 16) ? d_hi : d_lo;
  }
  // O = acc / (6 D) for E2M1 payloads (P and V each carry 1/6); FP8 payloads carry none
  const float inv = 1.0f / ((PV8 ? 1.0f : 6.0f) * Dfin);
  const size_t orow = ((size_t)bh * N + qrow) * D;
#pragma unroll
  for (int c = 0; c < D / 32; ++c) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col = 32 * c + 8 * g + 4 * h;
      const float o0 = O[c][4 * g] * inv, o1 = O[c][4 * g + 1] * inv;
      const float o2 = O[c][4 * g + 2] * inv, o3 = O[c][4 * g + 3] * inv;
      if (p.out_bf16) {
        typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
        const unsigned w0 = __builtin_bit_cast(unsigned, bf2{(__bf16)o0, (__bf16)o1});
        const unsigned w1 = __builtin_bit_cast(unsigned, bf2{(__bf16)o2, (__bf16)o3});
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(p.out) + orow + col) = uint2{w0, w1};
      } else {
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(p.out) + orow + col) = float4{o0, o1, o2, o3};
      }
    }
  }
  if constexpr (DUMP) {
    if (slot >= 0 && h == 0) {
      p.row_m[slot] = GUARD ? 0 : (int)Mref;
      p.row_d[slot] = Dfin;
    }
    if constexpr (CAUSAL) {
      // blocks past the workgroup's last query are never visited: code 0, no exponent
      if (slot >= 0) {
        for (int kb = 2 * nsteps + h; kb < N / 32; kb += 2) {
          *reinterpret_cast<POp*>(p.p_codes + (size_t)slot * (PV8 ? N : N / 2) + kb * (PV8 ? 32 : 16)) = POp{};
          p.block_exp[(size_t)slot * (N / 32) + kb] = (int16_t)-32768;
        }
      }
    }
  }
  if (p.lse != nullptr && h == 0) {
    // ln(sum_j 2^y_ij) of the represented operator: 2^ref * D / 6, with ref = M_i
    // (online) or R_i + L (guard, whose published bytes are shifted down by L)
    constexpr float kLn2 = 0.69314718f, kLn6 = 1.79175947f;
    const float ref = GUARD ? Rref + p.shift : Mref;
    // (FP8 route: D already carries the payload's 2^-7, and no 1/6)
    p.lse[(size_t)bh * N + qrow] = ref * kLn2 + (PV8 ? logf(Dfin) : logf(Dfin) - kLn6);
  }
  if (p.wg_clock != nullptr && tid == 0) {
    // shader-clock cycles and 100 MHz constant-clock ticks this workgroup was resident
    const unsigned long long clk1 = __builtin_amdgcn_s_memtime(), rt1 = __builtin_amdgcn_s_memrealtime();
    p.wg_clock[2 * blockIdx.x] = clk1 - clk0;
    p.wg_clock[2 * blockIdx.x + 1] = rt1 - rt0;
  }
}

template <int D, int NW, bool DUMP, int EX2, int VAR>
hipError_t launch_directp(const KParams& kp, hipStream_t stream) {
  hipLaunchKernelGGL((fwd_mxfp4_kernel<D, NW, DUMP, EX2, VAR>), dim3(kp.total), dim3(NW * 64), 0, stream, kp);
  return hipGetLastError();
}

// Every (D, NW, DUMP) variant of one EX2 density and reference variant.
#define FP4ATTN_DIRECTP_VARIANTS(MACRO, EX2, VAR) \
  MACRO(64, 4, false, EX2, VAR)                   \
  MACRO(64, 4, true, EX2, VAR)                    \
  MACRO(64, 8, false, EX2, VAR)                   \
  MACRO(64, 8, true, EX2, VAR)                    \
  MACRO(128, 4, false, EX2, VAR)                  \
  MACRO(128, 4, true, EX2, VAR)                   \
  MACRO(128, 8, false, EX2, VAR)                  \
  MACRO(128, 8, true, EX2, VAR)

#define FP4ATTN_DIRECTP_DECLARE(D, NW, DUMP, EX2, VAR) \
  extern template hipError_t launch_directp<D, NW, DUMP, EX2, VAR>(const KParams&, hipStream_t);
#define FP4ATTN_DIRECTP_DEFINE(D, NW, DUMP, EX2, VAR) \
  template hipError_t launch_directp<D, NW, DUMP, EX2, VAR>(const KParams&, hipStream_t);

}  // namespace directp_detail
}  // namespace fp4attn
