// Same-design BF16 attention forward: the in-house speed baseline for the
// paper's canonical speedup t_BF16 / t_FP4 (eq. canonical-speedup).
//
// Textbook softmax attention (eq. exact-attention) with the online recurrence
// (eq. online-recurrence) in base 2, on the skeleton of the MXFP4 forward:
// - transposed products S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_32x32x16_bf16,
//   so lane l owns query l % 32 in every accumulator and the row state is a
//   per-lane scalar; 32 queries per wave, NW waves per workgroup;
// - keys enter the S^T product permuted (key_of_row16) so that lane half h
//   holds keys 8h .. 8h+7 and 16+8h .. 16+8h+7 of each 32-key step, in order:
//   the bf16 probabilities it computes are already its P^T operand of the PV
//   product, with no cross-lane movement;
// - K/V tiles of 64 keys in a four-stage LDS ring filled three tiles ahead by
//   direct-to-LDS buffer loads: K in matrix-operand order, V in its natural
//   [key][d] layout (16-byte chunks XOR-swizzled by key), read as the V^T
//   operand by gfx950's transposing LDS read (ds_read_b64_tr_b16), so V is
//   taken as [B, H, N, d] like Q and K;
// - a two-deep software pipeline: while the vector ALU turns step g+1 into
//   probabilities, the matrix unit runs PV of step g and QK of step g+2;
// - an integer row reference with a lazy, exact power-of-two rescale (the
//   reference may lag the row maximum by up to 32 binades), and the denominator
//   from the same bf16 P operand on the matrix unit (an indicator-row
//   16x16x32 product), so it sums exactly the probabilities PV consumes;
// - the XCD-aware workgroup order of the MXFP4 forward, and its eight-wave
//   workgroups at d = 128 (two per CU at four waves per SIMD at d = 64).
#include "gfx950.hpp"
#include "launch.hpp"

namespace fp4attn {

namespace {

constexpr int kBN16 = 64;       // keys per LDS tile
constexpr int kStages16 = 4;    // LDS ring depth in tiles
constexpr float kTau16 = 32.0f;  // lazy rescale threshold in log2 units
constexpr float kLog2Ef = 1.4426950408889634f;

struct BParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  void* out;
  int N, n_qtiles, total;
  float sc;  // softmax_scale * log2(e)
};

template <int D>
struct BLayout {
  static constexpr int kCodes = (kBN16 / 32) * (D / 16) * 1024;  // K fragments [step][d chunk][lane][16 B]
  static constexpr int vCodes = kBN16 * D * 2;                   // V [key][d], swizzled 16-byte chunks
  static constexpr int kOff = 0;
  static constexpr int vOff = kCodes;
  static constexpr int stage = kCodes + vCodes;
};

// V tiles in LDS: key r's 16-byte chunk c (d = 8 c .. 8 c + 7) sits in slot
// c ^ swz(r) of its row.  A transposing read of one d block touches 8 rows
// (r % 16 = 8 h + 4 t + i / 4 over the lanes) and 4 chunks; the swizzle spreads
// those 32 pieces over all 64 banks, two per 16-byte bank group: for d = 128 (a
// row is 256 bytes) with the row's low two bits in the slot's high bits and its
// next two in the low bits; for d = 64 (two rows per 256 bytes) likewise with
// bit 1 of the row instead of its low two bits.
template <int D>
__device__ __forceinline__ int v_swizzle(int r) {
  return D == 128 ? 4 * (r & 3) + ((r >> 2) & 3) : 4 * ((r >> 1) & 1) + ((r >> 2) & 3);
}

// Key order of the S^T product within a 32-key step: operand row m = 8 g + 4 h + i
// holds key 16 (g / 2) + 8 h + 4 (g % 2) + i.  With the 32x32 accumulator layout
// (row 8 (r / 4) + 4 h + r % 4 in register r of lane half h), register r of lane
// half h then holds key 16 (r / 8) + 8 h + r % 8.
__device__ __forceinline__ int key_of_row16(int m) {
  return 16 * (m >> 4) + 8 * ((m >> 2) & 1) + 4 * ((m >> 3) & 1) + (m & 3);
}

// Direct-to-LDS copy of lane l's 16 bytes at byte soff + off of `rsrc` to LDS
// byte `lds` + 16 l (see the MXFP4 forward: not counted by the compiler, waited
// for with vm_wait; bytes past the buffer's end read as zero).
__device__ __forceinline__ void lds_copy16_b(unsigned lds, __amdgpu_buffer_rsrc_t rsrc, int soff, unsigned off) {
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(off), "s"(rsrc),
               "s"(__builtin_amdgcn_readfirstlane(soff)), "{m0}"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}
template <int n>
__device__ __forceinline__ void vm_wait_b() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n) : "memory");
}
__device__ __forceinline__ unsigned lds_address_b(const uint8_t* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_buffer_b(const void* base, int bytes) {
  const uint64_t a = (uint64_t)base;
  const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)a), hi = __builtin_amdgcn_readfirstlane((unsigned)(a >> 32));
  void* b = (void*)(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(b, (short)0, __builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

// One 64-key tile: K fragments in operand order (item i = one lane's 16 bytes
// of step s, d chunk c), then V rows in [key][d] order with the 16-byte chunk
// c of key r stored at chunk slot c ^ v_swizzle(r).  Thread tid copies items
// tid, tid + NT, ...; the 64 lanes of a wave copy 64 consecutive items.
template <int D, int NW>
struct TileCopy16 {
  using L = BLayout<D>;
  static constexpr int NT = NW * 64;
  static constexpr int nK = L::kCodes / 16;
  static constexpr int nV = L::vCodes / 16;
  static constexpr int kItems = nK + nV;
  static constexpr int kPerThread = kItems / NT;  // loads every wave issues per tile
  static_assert(kItems % NT == 0 && nK % NT == 0, "whole waves per operand");

  __amdgpu_buffer_rsrc_t buf[kPerThread];  // wave-uniform
  unsigned lds_off[kPerThread];            // wave-uniform
  unsigned off[kPerThread];                // this lane's byte offsets within a tile

  __device__ __forceinline__ void init(const uint16_t* kp, const uint16_t* vp, int N, int tid) {
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const __amdgpu_buffer_rsrc_t kbuf = make_buffer_b(kp, N * D * 2);
    const __amdgpu_buffer_rsrc_t vbuf = make_buffer_b(vp, N * D * 2);
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int item0 = wave * 64 + i * NT, item = item0 + lane;
      const bool is_k = i < nK / NT;  // compile-time
      buf[i] = is_k ? kbuf : vbuf;
      lds_off[i] = item0 * 16;
      if (is_k) {
        const int m = item & 63, rest = item >> 6;
        const int c = rest % (D / 16), s = rest / (D / 16);
        off[i] = ((32 * s + key_of_row16(m & 31)) * D + 16 * c + 8 * (m >> 5)) * 2;
      } else {
        const int p = item - nK, r = p / (D / 8), slot = p % (D / 8);
        off[i] = (r * D + 8 * (slot ^ v_swizzle<D>(r))) * 2;
      }
    }
  }

  // Fetch the tile of keys [key0, key0 + 64) into stage `st`.
  __device__ __forceinline__ void issue(uint8_t* st, int key0) const {
    const unsigned lds = lds_address_b(st);
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) lds_copy16_b(lds + lds_off[i], buf[i], key0 * D * 2, off[i]);
  }
};

__device__ __forceinline__ unsigned pack_bf16(float lo, float hi) {
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(unsigned, bf2{(__bf16)lo, (__bf16)hi});
}

// Four consecutive keys of one d column through the transposing LDS read: in each
// group of 16 lanes, lane j receives element j % 4 of the 8 bytes addressed by
// lane 4 e + j / 4 of its group, for e = 0..3.
__device__ __forceinline__ uint2 lds_read_tr16(const uint8_t* p) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  const v4s r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(p));
  return __builtin_bit_cast(uint2, r);
}

// Two waves per SIMD, except four-wave workgroups with d = 128, whose 128 KiB
// ring leaves room for one workgroup per CU, and eight-wave workgroups with
// d = 64, two per CU (64 KiB of LDS each) at four waves per SIMD (at most 128
// registers).
template <int D, int NW>
constexpr int kMinWaves16 = (D == 128 && NW == 4) ? 1 : ((D == 64 && NW == 8) ? 4 : 2);

template <int D, int NW, bool OUT_BF16>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(kMinWaves16<D, NW>, kMinWaves16<D, NW> > 2 ? 4 : 2))) void
fwd_bf16_kernel(const BParams p) {
  using L = BLayout<D>;
  constexpr int BM = NW * 32;
  __shared__ __attribute__((aligned(16))) uint8_t ring0[L::stage];
  __shared__ __attribute__((aligned(16))) uint8_t ring1[L::stage];
  __shared__ __attribute__((aligned(16))) uint8_t ring2[L::stage];
  __shared__ __attribute__((aligned(16))) uint8_t ring3[L::stage];
  static_assert(kStages16 == 4, "one array per ring stage");
  auto ring = [&](auto B_) -> uint8_t* {
    constexpr int b = decltype(B_)::value % kStages16;
    if constexpr (b == 0) return ring0;
    else if constexpr (b == 1) return ring1;
    else if constexpr (b == 2) return ring2;
    else return ring3;
  };

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, h = lane >> 5, lr = lane & 31;
  const int lin = xcd_remap(blockIdx.x, p.total);
  const int bh = lin / p.n_qtiles, qt = lin % p.n_qtiles;
  const int N = p.N;
  const int qrow = qt * BM + wave * 32 + lr;

  const uint16_t* kp = p.k + (size_t)bh * N * D;
  const uint16_t* vp = p.v + (size_t)bh * N * D;

  // Q^T operand (B of the S^T product), resident: lane l, d = 16 c + 8 h + [0, 8).
  v4i qf[D / 16];
  {
    const uint16_t* qr = p.q + ((size_t)bh * N + qrow) * D;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) qf[c] = *reinterpret_cast<const v4i*>(qr + 16 * c + 8 * h);
  }

  // Denominator operand (A of a 16x16x32 product).  Read as that product's B
  // operand, the P^T register of lane l is column l % 16 and k-block l / 16,
  // i.e. query l % 32's keys 8 (l / 32) .. +7 of a 16-key chunk: row 0 of this
  // indicator selects k-blocks 0 and 2 (query c), row 1 k-blocks 1 and 3 (query
  // c + 16), so one product per chunk yields every query's probability sum.
  const int ones_word = (lane == 0 || lane == 32 || lane == 17 || lane == 49) ? 0x3f803f80 : 0;  // bf16 1.0
  const v4i ones = {ones_word, ones_word, ones_word, ones_word};

  v16f O[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c) O[c] = v16f{};
  v4f Dacc = {};          // lane c < 16: register 0 = query c, register 1 = query c + 16
  float Mref = -1.0e6f;   // integer row reference (exact in fp32); no key seen yet
  float Mthr = Mref + kTau16;

  // The lane's part of its transposing V reads, one offset per d block cc and key
  // quarter t: lane i of group g = l / 16 reads key row 8 h + 4 t + i / 4 (plus a
  // multiple of 16, which leaves the swizzle unchanged) at d = 32 cc + 16 (g % 2) +
  // 4 (i % 4), i.e. chunk 4 cc + 2 (g % 2) + (i % 4) / 2, byte 8 (i % 2).
  const int gi = lane & 15, gg = (lane >> 4) & 1;
  unsigned v_lane[D / 32][2];
#pragma unroll
  for (int cc = 0; cc < D / 32; ++cc)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int r = 8 * h + 4 * t + gi / 4;
      v_lane[cc][t] = r * (2 * D) + 16 * ((4 * cc + 2 * gg + (gi & 3) / 2) ^ v_swizzle<D>(r)) + 8 * (gi & 1);
    }

  const int ntiles = N / kBN16;
  const int nsteps = 2 * ntiles;  // 32-key steps

  // S^T of 32-key step `sl` (0 or 1) of the tile held in `st`.
  auto qk = [&](const uint8_t* st, auto SL_, v16f& acc) {
    constexpr int sl = decltype(SL_)::value;
    v16f a = v16f{};
    static_for<D / 16>([&](auto C_) {
      constexpr int c = decltype(C_)::value;
      const v4i kf = *reinterpret_cast<const v4i*>(st + L::kOff + ((sl * (D / 16) + c) * 64 + lane) * 16);
      a = mfma_bf16_32x32x16(kf, qf[c], a);
    });
    acc = a;
  };

  // PV of step `s` (0 or 1) of the tile held in `st` and the denominator from the
  // same P^T operands.  V^T operand of chunk c, d block cc: lane l, d = 32 cc + l % 32,
  // keys 32 s + 16 c + 8 h + [0, 8), two transposing reads of four keys each.
  auto pv = [&](const uint8_t* st, auto S_, const v4i (&P)[2]) {
    constexpr int s = decltype(S_)::value;
    static_for<2>([&](auto C_) {
      constexpr int c = decltype(C_)::value;
      static_for<D / 32>([&](auto CC_) {
        constexpr int cc = decltype(CC_)::value;
        constexpr int o = (32 * s + 16 * c) * (2 * D);
        const uint2 lo = lds_read_tr16(st + L::vOff + o + v_lane[cc][0]);
        const uint2 hi = lds_read_tr16(st + L::vOff + o + v_lane[cc][1]);
        const v4i vf = {(int)lo.x, (int)lo.y, (int)hi.x, (int)hi.y};
        O[cc] = mfma_bf16_32x32x16(vf, P[c], O[cc]);
      });
      Dacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, ones), __builtin_bit_cast(v8bf, P[c]),
                                                     Dacc, 0, 0, 0);
    });
  };

  // Instruction order of one steady-state step (the region before the rescale
  // branch): the step's V^T reads first, the row-maximum chain while they land,
  // then every PV and denominator MFMA followed by a slice of the probabilities.
  constexpr int kStepMfma = 2 * (D / 32) + 2;
  auto schedule_step = [&]() {
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * (D / 32) * 2, 0);  // DS reads: V^T fragments
    __builtin_amdgcn_sched_group_barrier(0x002, 12, 0);                // VALU: row maximum
    static_for<kStepMfma>([&](auto) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                              // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, (40 + kStepMfma - 1) / kStepMfma, 0);  // probabilities
    });
  };

  // P = 2^(s log2(e) S - M) rounded to bf16 and packed into the two P^T chunk
  // operands (registers 8 c .. 8 c + 7 are keys 16 c + 8 h .. + 7).
  auto probabilities = [&](const v16f& S, v4i (&P)[2]) {
    const float nm = -Mref;
    static_for<2>([&](auto C_) {
      constexpr int c = decltype(C_)::value;
      unsigned w[4];
      static_for<4>([&](auto J_) {
        constexpr int j = decltype(J_)::value;
        const float e0 = __builtin_amdgcn_exp2f(fmaf(S[8 * c + 2 * j], p.sc, nm));
        const float e1 = __builtin_amdgcn_exp2f(fmaf(S[8 * c + 2 * j + 1], p.sc, nm));
        w[j] = pack_bf16(e0, e1);
      });
      P[c] = v4i{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
    });
  };

  // Step g's probabilities: row maximum over the step's 32 keys (16 per lane
  // half, then across the halves) and P with the current reference; only when
  // the maximum passes the reference by more than 32 binades (a wave-uniform, rare
  // branch) is the reference raised, O and the denominator rescaled exactly and
  // P recomputed, so the common path has no branch before the P work.
  auto softmax = [&](const v16f& S, v4i (&P)[2], auto SCHED_) {
    float m = fmaxf(fmaxf(S[0], S[1]), S[2]);
#pragma unroll
    for (int r = 3; r < 15; r += 2) m = fmaxf(fmaxf(m, S[r]), S[r + 1]);
    m = fmaxf(m, S[15]);
    unsigned ma = as_uint(m), mb = ma;
    swap_halves(ma, mb);
    const float y = fmaxf(as_float(ma), as_float(mb)) * p.sc;
    probabilities(S, P);
    // keep the probabilities next to the step's matrix work (emits nothing)
    asm volatile("" ::"v"(P[0]), "v"(P[1]));
    if constexpr (decltype(SCHED_)::value) schedule_step();
    if (__builtin_amdgcn_ballot_w64(y > Mthr)) {
      const float Mn = y > Mthr ? floorf(y) : Mref;
      const int sh = (int)(Mref - Mn);
#pragma unroll
      for (int c = 0; c < D / 32; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) O[c][r] = ldexpf(O[c][r], sh);
      Dacc[0] = ldexpf(Dacc[0], sh);
      Dacc[1] = ldexpf(Dacc[1], lane_read(sh, (lane + 16) & 63));  // query lane + 16
      Mref = Mn;
      Mthr = Mn + kTau16;
      probabilities(S, P);
    }
  };

  using Copy = TileCopy16<D, NW>;
  constexpr int kBatch = Copy::kPerThread;
  using I0 = std::integral_constant<int, 0>;
  Copy copy;
  copy.init(kp, vp, N, tid);
  copy.issue(ring(I0{}), 0);
  copy.issue(ring(std::integral_constant<int, 1>{}), kBN16);
  copy.issue(ring(std::integral_constant<int, 2>{}), 2 * kBN16);
  vm_wait_b<2 * kBatch>();  // tile 0 has landed
  __syncthreads();

  v16f SA, SB;
  v4i PA[2], PB[2];
  qk(ring(I0{}), std::integral_constant<int, 0>{}, SA);
  softmax(SA, PA, std::false_type{});
  qk(ring(I0{}), std::integral_constant<int, 1>{}, SA);

  // One step of the pipeline (see the MXFP4 forward): PV of step g, the
  // probabilities of step g+1, and QK of step g+2; j is the step's position in
  // its group of eight, TAIL marks the tail group.
  auto step = [&](auto J_, auto TAIL_, int g) {
    constexpr int j = decltype(J_)::value;
    constexpr bool tail = decltype(TAIL_)::value;
    constexpr int sl = j % 2;
    using b_cur = std::integral_constant<int, j / 2>;
    using b_nxt = std::integral_constant<int, j / 2 + 1>;
    using b_new = std::integral_constant<int, j / 2 + 3>;
    auto& S_in = (sl == 0) ? SA : SB;   // S^T of step g+1
    auto& S_out = (sl == 0) ? SB : SA;  // S^T of step g+2
    auto& P_cur = (sl == 0) ? PA : PB;
    auto& P_nxt = (sl == 0) ? PB : PA;
    const int t = g >> 1;
    pv(ring(b_cur{}), std::integral_constant<int, sl>{}, P_cur);
    if (!tail || g + 1 < nsteps) softmax(S_in, P_nxt, std::bool_constant<!tail>{});
    if constexpr (sl == 0) {
      vm_wait_b<kBatch>();  // tile t+1 has landed: only tile t+2's loads may be in flight
      __syncthreads();
      copy.issue(ring(b_new{}), (t + 3) * kBN16);
    }
    if (!tail || g + 2 < nsteps) {
      qk(ring(b_nxt{}), std::integral_constant<int, sl>{}, S_out);
      asm volatile("" ::"v"(S_out));
    }
  };

  int g0 = 0;
  for (; g0 + 8 <= nsteps - 2; g0 += 8) {
    static_for<8>([&](auto J_) { step(J_, std::false_type{}, g0 + decltype(J_)::value); });
  }
  static_for<10>([&](auto J_) {
    const int g = g0 + decltype(J_)::value;
    if (g < nsteps) step(J_, std::true_type{}, g);
  });
  vm_wait_b<0>();  // no copy may still be landing in LDS when the workgroup ends

  const float d_lo = lane_read(Dacc[0], lane & 15), d_hi = lane_read(Dacc[1], lane & 15);
  const float inv = 1.0f / ((lane & 16) ? d_hi : d_lo);
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
  bp.v = static_cast<const uint16_t*>(a.v);
  bp.out = a.out;
  bp.N = a.N;
  bp.sc = a.softmax_scale * kLog2Ef;
  const int bh = a.B * a.H;
  // d = 128: eight-wave (256-query) workgroups when they fill the chip (four
  // waves would run one wave per SIMD).  d = 64: eight-wave workgroups, two per
  // CU, from half a round of them on.
  const int64_t wide_wgs = a.N % 256 == 0 ? (int64_t)(a.N / 256) * bh : 0;
  const bool wide = a.d == 128 ? wide_wgs >= 256 : wide_wgs >= 128;
  const int BM = wide ? 256 : 128;
  bp.n_qtiles = a.N / BM;
  bp.total = bp.n_qtiles * bh;
  if (a.d == 128) return wide ? launch_b<128, 8>(bp, a.out_bf16, stream) : launch_b<128, 4>(bp, a.out_bf16, stream);
  return wide ? launch_b<64, 8>(bp, a.out_bf16, stream) : launch_b<64, 4>(bp, a.out_bf16, stream);
}

}  // namespace fp4attn
