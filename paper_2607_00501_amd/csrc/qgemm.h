// Q4/Q8 MFMA GEMM core shared by the prefill GEMM and the MoE grouped GEMMs.
//
// Y = A * W'^T with W' the group-32 Q4 (or, for the dense GEMM, Q8) weights
// dequantised inside the kernel (BaseRT Sec. 3.3: dequantisation in the matmul inner loop; Sec.
// 3.4: tiled GEMM for prefill).  Mapping on gfx950 (64-lane wavefronts,
// v_mfma_f32_32x32x16_f16):
//  * a workgroup has WN x WK wavefronts; wavefront (wn, wk) owns the BM x 64
//    output block whose 64 columns are one device-layout panel, over the
//    wk-th slice of the K steps (WK > 1: split-K inside the workgroup, in
//    every mode; the partial sums meet in LDS in a fixed order).  One 64-deep
//    K step of its weights is two 1 KiB contiguous chunk rows (Q8: two
//    2 KiB chunks, each two 1 KiB halves of 16 k);
//  * loads go global -> LDS by DMA (global_load_lds_dwordx4: lane l of an
//    instruction lands at M0 + 16 l, 1 KiB per instruction), with no staging
//    registers: the activation tile of each K slice (BM x 64 fp16, shared by
//    the WN wavefronts of the slice) and, for multi-wavefront tiles whose
//    stages fit, each wavefront's two chunk rows verbatim plus their scales.
//    One-wavefront split-K tiles load the weights into registers instead.
//    LDS activation rows are 128 B; 16-byte chunk c of row r sits at
//    position c ^ ((r >> 1) & 7), so the A-fragment reads of 16 consecutive
//    rows touch all 64 banks;
//  * each wavefront dequantises its own B fragments in registers, once per
//    workgroup.  The 16-deep k block an MFMA lane half covers is relabelled
//    (A and B agree, so the sum is unchanged): in substep s of group c, lane
//    half h takes k = 32c + 16h + 8s + 0..7.  Lane l then needs two
//    consecutive dwords of row l%32 (column half 0) and of row 32 + l%32
//    (column half 1) (Q8: 16 bytes, the row's half h): no cross-lane
//    permute.  Q4: v_and_or_b32 + one packed fp16 add (or an exact fma for
//    the nibbles at bits 4-7) + v_pk_mul_f16; Q8: v_perm_b32 + one packed
//    add + v_pk_mul_f16; both give fp16_RNE(s*q) exactly.  A fragments and
//    dequantised B of the next substep are produced while the current MFMAs
//    run;
//  * loads run DEPTH (2-3) K steps ahead into DEPTH + 1 LDS stages / register
//    slots (2 stages, one step ahead, where LDS is short), so a load always
//    targets a slot whose step is already consumed (no loop-carried register
//    copies).  Each K step waits for exactly its own loads and then passes
//    one barrier.  Out-of-range rows, columns and K steps (also the
//    prefetches past the last step) read clamped (valid) addresses with
//    their scales forced to zero, so the loads carry no branches;
//  * modes: kDense (rows m0.., plain row-major A and Y); kMoeGateUp (rows of
//    one expert's bucket, A rows gathered through the assignment
//    permutation, each wavefront streams the gate and the up panel of the
//    same columns and the epilogue writes fp16 silu(gate) * up); kMoeDown
//    (A = the fp16 h rows of the bucket, the epilogue scales by the
//    assignment's gate weight and scatters the row, in fp16, to its
//    assignment slot).
//    MoE workgroups find their (expert, row tile) from the per-expert counts
//    on the device, so no host synchronisation is needed.
#pragma once

#include <type_traits>
#include <utility>

#include "qm_internal.h"

namespace qm {

enum class QgMode { kDense = 0, kMoeGateUp = 1, kMoeDown = 2 };

struct QgemmArgs {
  const uint8_t* q;  const uint16_t* s;    // dense weights; MoE gate or down experts
  const uint8_t* q2; const uint16_t* s2;   // MoE up experts (kMoeGateUp)
  const uint16_t* a;                       // A rows: X (dense, gate/up) or h (down)
  float* y;                                // dense output [M][N]
  int64_t M, N, K;                         // MoE: M = number of assignments
  const int32_t* counts;
  const int32_t* offsets;
  const int32_t* sorted_assign;
  const float* topk_w;
  const int32_t* topk_ids;                 // MoE: expert of each assignment (checked by kMoeDown)
  uint16_t* h;                             // kMoeGateUp output [M][N] fp16 (bucket order)
  uint16_t* yp;                            // kMoeDown output [M][N] fp16 (assignment order)
  int32_t n_experts, top_k;
  int64_t tiles;                           // MoE: bound on the number of (expert, row tile) pairs
  // kDense: gcount matrices with one K and a shared A, side by side in the
  // panel index space (matrix i owns panels [gpanel[i], gpanel[i+1]));
  // each wavefront picks its matrix.  A single GEMM is a group of one.
  int32_t gcount;
  int32_t gpanel[kGemmGroupMax + 1];
  const uint8_t* gq[kGemmGroupMax];
  const uint16_t* gs[kGemmGroupMax];
  float* gy[kGemmGroupMax];
  int64_t gn[kGemmGroupMax];
};

namespace qg {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kBK = 64;                 // K per step (two quantisation groups)
constexpr int kMoeChunkTiles = 4;       // MoE row tiles per XCD chunk

// s_waitcnt vmcnt(N) with expcnt and lgkmcnt left free (gfx9 encoding:
// vmcnt[3:0] in bits 3:0 and vmcnt[5:4] in bits 15:14).
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// vm_wait<BASE + live * PER>() for a wavefront-uniform live in [0, L...]
// (s_waitcnt takes an immediate: one scalar branch per candidate).
template <int BASE, int PER, int... L>
__device__ __forceinline__ void vm_wait_live(int live, std::integer_sequence<int, L...>) {
  ((live == L ? vm_wait<BASE + L * PER>() : void()), ...);
}

// 16 bytes per lane from global memory straight into LDS: lane l of the
// wavefront writes lds_dst + 16 l (lds_dst is wavefront-uniform and goes
// to M0).  Issued as inline asm so that the compiler's wait-count tracking
// does not see it: with an LDS DMA pending, that tracking would wait for
// every outstanding load (vmcnt 0) before the next use of any loaded
// register.  The hardware still counts it in vmcnt; the kernel waits for it
// explicitly (vm_wait), and every later wait the compiler computes stays
// conservative.
__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<size_t>((const void __attribute__((address_space(3)))*)p));
}
template <bool NT = false>
__device__ __forceinline__ void lds_dma16(const void* src, const void* lds_dst) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" : : "v"(src), "s"(lds_address(lds_dst))
                 : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "s"(lds_address(lds_dst))
                 : "memory", "m0");
}
// 4 bytes per lane, lane l to lds_dst + 4 l.
template <bool NT = false>
__device__ __forceinline__ void lds_dma4(const void* src, const void* lds_dst) {
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off nt" : : "v"(src), "s"(lds_address(lds_dst))
                 : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" : : "v"(src), "s"(lds_address(lds_dst))
                 : "memory", "m0");
}

// Dequantisation constants held in registers: the masks 0x000F000F and
// 0x00F000F0 in VGPRs and the fp16 magic 0x6400_6400 in an SGPR, so that
// (d & mask) | magic selects to one v_and_or_b32 (gfx9 VOP3 takes no literal
// operand).  The empty asm makes the values opaque once, outside the loops.
struct DequantRegs {
  uint32_t m0, m1, magic_s;
  __device__ DequantRegs() : m0(0x000F000Fu), m1(0x00F000F0u), magic_s(0x64006400u) {
    asm volatile("" : "+v"(m0), "+v"(m1));
    asm volatile("" : "+s"(magic_s));
  }
};

// 8 offset-binary nibbles of one device-layout dword (k order 0,2,4,6 |
// 1,3,5,7) -> 8 fp16 fp16_RNE(s*q) in natural k order.  Nibbles at bits 0-3
// (and 16-19) give the fp16 1024 + u, so q = x - 1032; nibbles at bits 4-7
// (20-23) give 1024 + 16u, so q = x/16 - 72, one exact fma (x/16 is exact
// and q is a small integer).  Bits 8-15 take one shift and the same steps.
__device__ inline half8v dequant_dword(uint32_t d, half2v s2, const DequantRegs& c) {
  const half2v b1 = {(_Float16)1032.0f, (_Float16)1032.0f};
  const half2v r16 = {(_Float16)0.0625f, (_Float16)0.0625f};
  const half2v b16 = {(_Float16)-72.0f, (_Float16)-72.0f};
  const uint32_t d8 = d >> 8;
  const half2v q01 = __builtin_bit_cast(half2v, (d & c.m0) | c.magic_s) - b1;
  const half2v q23 = __builtin_elementwise_fma(__builtin_bit_cast(half2v, (d & c.m1) | c.magic_s), r16, b16);
  const half2v q45 = __builtin_bit_cast(half2v, (d8 & c.m0) | c.magic_s) - b1;
  const half2v q67 = __builtin_elementwise_fma(__builtin_bit_cast(half2v, (d8 & c.m1) | c.magic_s), r16, b16);
  const half2v v0 = q01 * s2, v1 = q23 * s2, v2 = q45 * s2, v3 = q67 * s2;
  return half8v{v0[0], v0[1], v1[0], v1[1], v2[0], v2[1], v3[0], v3[1]};
}

// Q8 constants: v_perm_b32 selectors in VGPRs and the byte 0x64 repeated in
// an SGPR (a VOP3 takes no literal and at most one scalar operand).
struct DequantRegsQ8 {
  uint32_t sel_lo, sel_hi, magic_s;
  __device__ DequantRegsQ8() : sel_lo(0x04010400u), sel_hi(0x04030402u), magic_s(0x64646464u) {
    asm volatile("" : "+v"(sel_lo), "+v"(sel_hi));
    asm volatile("" : "+s"(magic_s));
  }
};

// 8 offset-binary bytes u = q + 128 of the Q8 device layout (two dwords,
// natural k order) -> 8 fp16 fp16_RNE(s*q).  v_perm_b32 puts bytes 0, 1
// (or 2, 3) of a dword under the fp16 high byte 0x64, giving 1024 + u
// exactly; one packed subtract of 1152 leaves q, and v_pk_mul_f16 scales.
__device__ inline half8v dequant_q8(uint32_t d0, uint32_t d1, half2v s2, const DequantRegsQ8& c) {
  const half2v b = {(_Float16)1152.0f, (_Float16)1152.0f};
  const half2v q01 = __builtin_bit_cast(half2v, __builtin_amdgcn_perm(c.magic_s, d0, c.sel_lo)) - b;
  const half2v q23 = __builtin_bit_cast(half2v, __builtin_amdgcn_perm(c.magic_s, d0, c.sel_hi)) - b;
  const half2v q45 = __builtin_bit_cast(half2v, __builtin_amdgcn_perm(c.magic_s, d1, c.sel_lo)) - b;
  const half2v q67 = __builtin_bit_cast(half2v, __builtin_amdgcn_perm(c.magic_s, d1, c.sel_hi)) - b;
  const half2v v0 = q01 * s2, v1 = q23 * s2, v2 = q45 * s2, v3 = q67 * s2;
  return half8v{v0[0], v0[1], v1[0], v1[1], v2[0], v2[1], v3[0], v3[1]};
}

// Shift left by SH (right for negative SH); SH is a constant after unrolling.
__device__ __forceinline__ uint32_t shift_by(uint32_t v, int sh) { return sh >= 0 ? v << sh : v >> -sh; }

// Bit-plane formats, substep s of a lane's 16 codes (k = 16h + 8s .. +7 of
// the group, natural order) -> 8 fp16 fp16_RNE(s*q).
//  Q5 / Q6: nibble dword nd (Q4 order) plus the high part of u: Q5 from the
//  bit dword hb (already shifted right by 8h, so pair p of the 8 lies at
//  bits p and 16 + p), Q6 from the crumb dword cw (pair p at 2p, 16 + 2p).
//  The high bits join the Q4 fp16-magic lanes at mantissa bit 4 (lanes of
//  1024 + u) or 8 (lanes of 1024 + 16u); both stay exact (16u <= 1008).
template <int FMT>
__device__ inline half8v dequant_nib_hi(uint32_t nd, uint32_t hi_w, int s, half2v s2, const DequantRegs& c) {
  constexpr int bias = FMT == QM_Q5_G32 ? 16 : 32;
  const half2v b1 = {(_Float16)(1024 + bias), (_Float16)(1024 + bias)};
  const half2v r16 = {(_Float16)0.0625f, (_Float16)0.0625f};
  const half2v b16 = {(_Float16)(-64 - bias), (_Float16)(-64 - bias)};
  auto hi = [&](int pair, int T) __attribute__((always_inline)) {
    if constexpr (FMT == QM_Q5_G32) return shift_by(hi_w, T - (4 * s + pair)) & ((1u << T) | (1u << (T + 16)));
    else return shift_by(hi_w, T - 2 * (4 * s + pair)) & ((3u << T) | (3u << (T + 16)));
  };
  const uint32_t d8 = nd >> 8;
  const half2v q01 = __builtin_bit_cast(half2v, ((nd & c.m0) | c.magic_s) | hi(0, 4)) - b1;
  const half2v q23 = __builtin_elementwise_fma(__builtin_bit_cast(half2v, ((nd & c.m1) | c.magic_s) | hi(1, 8)), r16, b16);
  const half2v q45 = __builtin_bit_cast(half2v, ((d8 & c.m0) | c.magic_s) | hi(2, 4)) - b1;
  const half2v q67 = __builtin_elementwise_fma(__builtin_bit_cast(half2v, ((d8 & c.m1) | c.magic_s) | hi(3, 8)), r16, b16);
  const half2v v0 = q01 * s2, v1 = q23 * s2, v2 = q45 * s2, v3 = q67 * s2;
  return half8v{v0[0], v0[1], v1[0], v1[1], v2[0], v2[1], v3[0], v3[1]};
}
//  Q2 / Q3: crumb dword cw of the lane's 16 codes (pair p of substep s at
//  bits 2(4s + p), 16 + 2(4s + p)); masked in place it gives 1024 + 4^p u
//  (after a shift by 8 for s = 1), and one exact fma x * 4^-p - (1024 * 4^-p
//  + bias) leaves q.  Q3 adds its bit (hb, shifted right by 8h) at bit
//  2p + 2 of the same lanes (4^3 * 7 = 448 keeps the value in [1024, 2048)).
template <int FMT>
__device__ inline half8v dequant_crumb(uint32_t cw, uint32_t hb, int s, half2v s2, const DequantRegs& c) {
  constexpr int bias = FMT == QM_Q2_G32 ? 2 : 4;
  const uint32_t src = s ? cw >> 8 : cw;
  half2v q[4];
#pragma unroll
  for (int pr = 0; pr < 4; ++pr) {
    uint32_t x = (src & (0x00030003u << (2 * pr))) | c.magic_s;
    if constexpr (FMT == QM_Q3_G32) {
      const int T = 2 * pr + 2;
      x |= shift_by(hb, T - (4 * s + pr)) & ((1u << T) | (1u << (T + 16)));
    }
    const _Float16 r = (_Float16)(1.0f / static_cast<float>(1 << (2 * pr)));
    const _Float16 b = (_Float16)(-(1024.0f / static_cast<float>(1 << (2 * pr))) - bias);
    q[pr] = __builtin_elementwise_fma(__builtin_bit_cast(half2v, x), half2v{r, r}, half2v{b, b}) * s2;
  }
  return half8v{q[0][0], q[0][1], q[1][0], q[1][1], q[2][0], q[2][1], q[3][0], q[3][1]};
}

// Wavefront 0 maps the workgroup's linear tile index to (expert, row tile)
// in expert order, with ceil(count / BM) tiles per expert.  Expert -1 when
// the index lies beyond the last tile.
__device__ inline void find_tile(const int32_t* counts, int E, int BM, int bx, int* sh_e, int* sh_tile) {
  if (threadIdx.x == 0) *sh_e = -1;
  __syncthreads();
  if ((threadIdx.x >> 6) == 0) {
    const int lane = threadIdx.x & 63;
    int running = 0;
    for (int b0 = 0; b0 < E; b0 += 64) {
      const int e = b0 + lane;
      const int t = e < E ? (counts[e] + BM - 1) / BM : 0;
      int incl = t;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int o = __shfl_up(incl, d);
        if (lane >= d) incl += o;
      }
      const int excl = running + incl - t;
      if (t > 0 && bx >= excl && bx < excl + t) {
        *sh_e = e;
        *sh_tile = bx - excl;
      }
      running += __shfl(incl, 63);
    }
  }
  __syncthreads();
}

template <int BM, int WN, int WK, QgMode MODE, int DEPTH, int FMT>
struct Cfg {
  static constexpr bool kQ8 = FMT == QM_Q8_G32;
  static constexpr bool kPlanes = FMT == QM_Q2_G32 || FMT == QM_Q3_G32 || FMT == QM_Q5_G32 || FMT == QM_Q6_G32;
  // F16 / BF16 weights: no codes, no scales; a lane's 8 k of a substep are
  // one 16-byte quarter of its row (BF16 converted to fp16 in registers).
  static constexpr bool kFloat = FMT == QM_F16 || FMT == QM_BF16;
  static_assert(FMT == QM_Q4_G32 || kQ8 || kPlanes || kFloat, "one of the eight weight formats");
  static constexpr int kChunkBytes = chunk_block_bytes(FMT);      // one group of a 64-row panel
  // B words a lane holds per group and column half: Q4 two nibble dwords,
  // Q8 four byte dwords, Q5/Q6 two nibble dwords + one high-plane dword,
  // Q3 one crumb + one bit dword, Q2 one crumb dword; and the global loads
  // (planes) behind them.
  static constexpr int kLW = FMT == QM_Q4_G32 ? 2 : kQ8 ? 4 : FMT == QM_Q2_G32 ? 1 : FMT == QM_Q3_G32 ? 2 : 3;
  static constexpr int kPlaneLoads = FMT == QM_Q3_G32 || FMT == QM_Q5_G32 || FMT == QM_Q6_G32 ? 2 : 1;
  static constexpr int kDwords = 2 * kLW;                         // B dwords per lane, column half and K step
  static constexpr int kPieces16 = kChunkBytes / 1024, kPieces4 = kChunkBytes % 1024 / 256;
  static constexpr bool kDual = MODE == QgMode::kMoeGateUp;
  static constexpr int kNB = kDual ? 2 : 1;                      // weight matrices per wavefront
  static constexpr int kThreads = WN * WK * 64;
  static constexpr int kSliceThreads = WN * 64;
  static constexpr int kTM = BM / 32;
  static constexpr int kALoads = BM * (kBK / 8) / kSliceThreads;
  static_assert(kALoads >= 1 && BM * (kBK / 8) % kSliceThreads == 0, "A tile split");
  static_assert(DEPTH >= 2 && DEPTH <= 3, "K steps of loads in flight");
  static constexpr int kSlots = DEPTH + 1;                       // slots of B (registers or LDS)
  // LDS stage: the A tiles of the WK slices (BM rows x 128 B each), then,
  // when B also goes through LDS, per wavefront and weight matrix the two
  // code chunks and their 2 x 64 scales (Q4 2304 B, Q8 4352 B).  B goes through LDS
  // for multi-wavefront slices whose DEPTH + 1 stages fit in 80 KiB (two
  // workgroups per CU); otherwise B is loaded into registers.
  static constexpr int kAStageBytes = WK * BM * kBK * 2;
  static constexpr int kBMatBytes = 2 * kChunkBytes + 256;
  static constexpr int kBWaveBytes = kNB * kBMatBytes;
  static constexpr bool kBLds = !kFloat && WN > 1 && kSlots * (kAStageBytes + WN * WK * kBWaveBytes) <= 80 * 1024;
  static constexpr int kStageBytes = kAStageBytes + (kBLds ? WN * WK * kBWaveBytes : 0);
  // A LDS stages: DEPTH + 1 (A loaded DEPTH steps ahead, like B) when they
  // fit in 48 KiB or B goes through LDS, else 2 (A loaded one step ahead),
  // so that two or more workgroups share a CU.
  static constexpr int kAStages = (kBLds || kSlots * kAStageBytes <= 48 * 1024) ? kSlots : 2;
  static constexpr int kADist = kAStages - 1;
  // Global loads of one K step issued by one wavefront: A row groups, then
  // per weight matrix either the code chunks in 1 KiB pieces + 1 scale
  // block (LDS DMA) or 2 chunks x 2 column halves of codes and of scales
  // (registers).
  static constexpr int kBLoads = kBLds ? kNB * (2 * (kPieces16 + kPieces4) + 1)
                                : kFloat ? kNB * 2 * 2 * 2 : kNB * 2 * 2 * (kPlaneLoads + 1);
  // Split-K partial sums of slices 1..WK-1, in halves (fp32 = 2 halves).
  static constexpr int kRedHalves = (WK - 1) * WN * kTM * 2 * kNB * 16 * 64 * 2;
  static constexpr int kLdsHalves =
      kAStages * kStageBytes / 2 > kRedHalves ? kAStages * kStageBytes / 2 : kRedHalves;
  static_assert(kAStages == kSlots || (kAStages == 2 && DEPTH == 2), "A stage schedule");
};

template <int BM, int WN, int WK, QgMode MODE, int DEPTH, bool NT, int FMT>
__device__ __forceinline__ void qgemm_body(const QgemmArgs& p) {
  using C = Cfg<BM, WN, WK, MODE, DEPTH, FMT>;
  constexpr bool Q8 = C::kQ8, PL = C::kPlanes;
  constexpr int CB = C::kChunkBytes, MB = C::kBMatBytes, LW = C::kLW;
  constexpr int NB = C::kNB;
  __shared__ __attribute__((aligned(16))) uint16_t lds[C::kLdsHalves];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wavefront-uniform (SGPR)
  const int wk = wave / WN, wn = wave % WN;
  const int64_t K = p.K, N = p.N;
  const int G = static_cast<int>(K / kGroup);
  const int KT = (G + 1) / 2;
  const int KTs = (KT + WK - 1) / WK;                      // K steps per slice
  const int kt0 = wk * KTs;
  const int64_t npad = padded_rows(N);

  // Rows of this workgroup.
  int64_t row0 = 0;
  int rows = 0;
  int expert = 0;
  int64_t col_block;
  if constexpr (MODE == QgMode::kDense) {
    row0 = static_cast<int64_t>(blockIdx.y) * BM;
    rows = static_cast<int>(min<int64_t>(BM, p.M - row0));
    col_block = blockIdx.x;
  } else {
    // 1-D grid over (row tile, column block) units, row-tile major, dealt to
    // the XCDs in chunks of kMoeChunkTiles row tiles: the row tiles of one
    // expert (same weight panels) and the column blocks of one tile (same A
    // rows) mostly share an L2.
    const int64_t ny = (npad + 64 * WN - 1) / (64 * WN);
    const int64_t u = xcd_chunked(blockIdx.x, kMoeChunkTiles * ny);
    if (u >= p.tiles * ny) return;                        // whole workgroup, before any barrier
    __shared__ int sh_e, sh_tile;
    find_tile(p.counts, p.n_experts, BM, static_cast<int>(u / ny), &sh_e, &sh_tile);
    expert = __builtin_amdgcn_readfirstlane(sh_e);
    if (expert < 0) return;
    row0 = p.offsets[expert] + static_cast<int64_t>(__builtin_amdgcn_readfirstlane(sh_tile)) * BM;
    rows = static_cast<int>(min<int64_t>(BM, p.offsets[expert + 1] - row0));
    col_block = u % ny;
  }
  // The wavefront's matrix (kDense groups) and its first output column.
  const uint8_t* mq = p.q;
  const uint16_t* ms = p.s;
  float* my = p.y;
  int64_t mN = N;
  int64_t n_wave = col_block * (64 * WN) + 64 * wn;
  bool cols_ok = n_wave < npad;
  if constexpr (MODE == QgMode::kDense) {
    const int gp = static_cast<int>(col_block * WN + wn);  // panel in the group's index space
    mq = p.gq[0]; ms = p.gs[0]; my = p.gy[0]; mN = p.gn[0];
    int first = 0;
#pragma unroll
    for (int j = 1; j < kGemmGroupMax; ++j) {
      const bool in = j < p.gcount && gp >= p.gpanel[j];
      mq = in ? p.gq[j] : mq;
      ms = in ? p.gs[j] : ms;
      my = in ? p.gy[j] : my;
      mN = in ? p.gn[j] : mN;
      first = in ? p.gpanel[j] : first;
    }
    n_wave = static_cast<int64_t>(gp - first) * kPanel;
    cols_ok = gp < p.gpanel[p.gcount];
  }
  const int64_t mnpad = padded_rows(mN);
  // kMoeDown: assignment id and gate weight of each row of the tile, staged
  // once in LDS for the epilogue (published by the barrier before the first
  // loads).
  __shared__ int64_t row_asg[MODE == QgMode::kMoeDown ? BM : 1];
  __shared__ float row_w[MODE == QgMode::kMoeDown ? BM : 1];
  if constexpr (MODE == QgMode::kMoeDown) {
    for (int r = tid; r < BM; r += C::kThreads) {
      const int64_t asg = p.sorted_assign[row0 + min(r, rows - 1)];
      row_asg[r] = asg;
      // An assignment whose bucket is not the expert topk_ids names gets a
      // NaN weight, so its token's output row is NaN (no host round trip).
      row_w[r] = p.topk_ids[asg] == expert ? p.topk_w[asg] : __builtin_nanf("");
    }
  }

  // A: instruction i of wavefront wn fills LDS row group g = i * WN + wn
  // (rows 8g .. 8g+7 of the stage); lane l lands at row 8g + l/8, position
  // l%8, i.e. it fetches logical chunk (l%8) ^ ((row >> 1) & 7) of that row
  // (rows clamped to the tile).
  const uint16_t* a_src[C::kALoads];
  int a_col[C::kALoads];
#pragma unroll
  for (int i = 0; i < C::kALoads; ++i) {
    const int row = 8 * (i * WN + wn) + (lane >> 3);
    a_col[i] = ((lane & 7) ^ ((row >> 1) & 7)) * 8;
    const int64_t r = row0 + min(row, rows - 1);
    int64_t src_row = r;
    if constexpr (MODE == QgMode::kMoeGateUp) src_row = p.sorted_assign[r] / p.top_k;
    a_src[i] = p.a + src_row * K;
  }
  // B: lane l reads dwords 2(l/32), 2(l/32)+1 of panel rows l%32 and
  // 32 + l%32 (Q8: the 16 bytes of half l/32 of those rows), clamped to a
  // real panel.  The matrix, expert and panel bases are wavefront-uniform;
  // the lane part is a 32-bit offset.
  const int64_t panel = (cols_ok ? n_wave : mnpad - kPanel) / kPanel;
  const int64_t mat_q = npad / kPanel * G * CB, mat_s = npad * G;   // bytes / scales of one matrix (MoE)
  const uint8_t* b_q[NB];
  const uint16_t* b_s[NB];
  b_q[0] = mq + expert * mat_q + panel * G * CB;
  b_s[0] = C::kFloat ? ms : ms + expert * mat_s + panel * G * kPanel;   // float weights: no scales (null)
  if constexpr (NB == 2) {
    b_q[1] = p.q2 + expert * mat_q + panel * G * CB;
    b_s[1] = C::kFloat ? p.s2 : p.s2 + expert * mat_s + panel * G * kPanel;
  }
  const uint32_t bq_lane = Q8 ? (lane & 31) * 16 + (lane >> 5) * 1024 : (lane & 31) * 16 + (lane >> 5) * 8;
  const uint32_t bs_lane = lane & 31;

  // DEPTH + 1 slots of raw B operands (registers, or LDS stages when B
  // goes through LDS) and kAStages LDS stages of A; step t lives in slot
  // t % (DEPTH + 1), always indexed by constants.  rb / rs are used only
  // when B is loaded into registers.
  constexpr int NS = C::kSlots;
  using BVec = std::conditional_t<Q8, u32x4, u32x2>;
  BVec rb[NS][NB][2][2];                                   // [slot][matrix][chunk][column half]
  uint32_t rw[NS][NB][2][2][LW];                           // the same for the bit-plane formats
  u32x4 rf[C::kFloat ? NS : 1][NB][2][2][2];               // F16/BF16: [..][column half][substep] quarters
  uint32_t rs[NS][NB][2][2];
  char* const lds_b = reinterpret_cast<char*>(lds);
  // A tile of this slice in stage st; B region of this wavefront in stage st.
  auto a_tile = [&](int st) __attribute__((always_inline)) { return lds_b + st * C::kStageBytes + wk * BM * 2 * kBK; };
  auto b_region = [&](int st) __attribute__((always_inline)) {
    return lds_b + st * C::kStageBytes + C::kAStageBytes + wave * C::kBWaveBytes;
  };
  auto load_a = [&](int st, int step) __attribute__((always_inline)) {
    const int kt = kt0 + step;
    char* tile = a_tile(st);
#pragma unroll
    for (int i = 0; i < C::kALoads; ++i) {
      const int k = min(kt * kBK + a_col[i], static_cast<int>(K) - 8);
      lds_dma16(a_src[i] + k, tile + (i * WN + wn) * 1024);
    }
  };
  auto load_b = [&](auto slot, int step) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot)::value;
    const int kt = kt0 + step;
    if constexpr (C::kBLds) {
      // Per matrix: the two code chunks verbatim in 1 KiB pieces, then
      // their scales (lanes 0-31: chunk 0, lanes 32-63: chunk 1; 4 B = 2
      // scales a lane).
      char* reg = b_region(sl);
      const int gs1 = min(2 * kt + (lane >> 5), G - 1);
#pragma unroll
      for (int j = 0; j < NB; ++j) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int gc = min(2 * kt + c, G - 1);
#pragma unroll
          for (int piece = 0; piece < C::kPieces16; ++piece)
            lds_dma16<NT>(b_q[j] + static_cast<int64_t>(gc) * CB + piece * 1024 + lane * 16,
                          reg + j * MB + c * CB + piece * 1024);
#pragma unroll
          for (int piece = 0; piece < C::kPieces4; ++piece)          // 256-byte tails (bit-plane formats)
            lds_dma4<NT>(b_q[j] + static_cast<int64_t>(gc) * CB + C::kPieces16 * 1024 + piece * 256 + lane * 4,
                         reg + j * MB + c * CB + C::kPieces16 * 1024 + piece * 256);
        }
        lds_dma4<NT>(b_s[j] + static_cast<int64_t>(gs1) * kPanel + 2 * (lane & 31), reg + j * MB + 2 * CB);
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int gc = min(2 * kt + c, G - 1);
        const uint8_t* bq = b_q[j] + static_cast<int64_t>(gc) * CB;
        if constexpr (C::kFloat) {
          // Row 32h + l%32: quarter 2(l/32) + s holds its k = 16(l/32) + 8s .. + 7.
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int sub = 0; sub < 2; ++sub) {
              const u32x4* qa = reinterpret_cast<const u32x4*>(bq + (2 * (lane >> 5) + sub) * 1024 +
                                                               16 * (32 * h + (lane & 31)));
              rf[C::kFloat ? sl : 0][j][c][h][sub] = NT ? __builtin_nontemporal_load(qa) : *qa;
            }
          continue;
        }
        const uint16_t* bs = b_s[j] + static_cast<int64_t>(gc) * kPanel;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint16_t* sa = bs + bs_lane + 32 * h;
          if constexpr (PL) {
            // Row 32h + l%32, lane half l/32: the planes of the bit-plane
            // formats (plain loads; these tiles are not built with NT).
            const int row = 32 * h + (lane & 31), lh = lane >> 5;
            uint32_t* w = rw[sl][j][c][h];
            if constexpr (FMT == QM_Q5_G32 || FMT == QM_Q6_G32) {
              const u32x2 nb = *reinterpret_cast<const u32x2*>(bq + row * 16 + 8 * lh);
              w[0] = nb.x; w[1] = nb.y;
              w[2] = FMT == QM_Q5_G32 ? *reinterpret_cast<const uint32_t*>(bq + 1024 + row * 4)
                                      : *reinterpret_cast<const uint32_t*>(bq + 1024 + row * 8 + 4 * lh);
            } else {
              w[0] = *reinterpret_cast<const uint32_t*>(bq + row * 8 + 4 * lh);
              if constexpr (FMT == QM_Q3_G32) w[1] = *reinterpret_cast<const uint32_t*>(bq + 512 + row * 4);
            }
            rs[sl][j][c][h] = *sa;
            continue;
          }
          const BVec* qa = reinterpret_cast<const BVec*>(bq + bq_lane + h * 512);
          if constexpr (NT) {
            rb[sl][j][c][h] = __builtin_nontemporal_load(qa);
            rs[sl][j][c][h] = __builtin_nontemporal_load(sa);
          } else {
            rb[sl][j][c][h] = *qa;
            rs[sl][j][c][h] = *sa;
          }
        }
      }
  };
  // Scale validity of step t's chunk c, applied when the step is consumed
  // (a select at load time would wait for the load to land).
  auto scale_ok = [&](int t, int c) __attribute__((always_inline)) {
    const int kt = kt0 + t;
    return cols_ok && 2 * kt + c < G && kt < KT;
  };
  // The A stages of a K slice are written (by LDS DMA) and read only by the
  // slice's WN wavefronts.  Each wavefront first waits for its own DMA of the
  // step (wait_a); a plain s_barrier then publishes every wavefront's part.
  // No memory fence: a workgroup fence would also wait for the loads of the
  // later steps still in flight.  The empty asm statements keep the compiler
  // from moving LDS accesses across the barrier.  A one-wavefront slice
  // needs no barrier.
  auto slice_sync = [&]() __attribute__((always_inline)) {
    asm volatile("" ::: "memory");
    if constexpr (WN > 1) __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  const std::conditional_t<Q8, DequantRegsQ8, DequantRegs> dq;
  float16v acc[C::kTM][2 * NB];
#pragma unroll
  for (int a = 0; a < C::kTM; ++a)
#pragma unroll
    for (int b = 0; b < 2 * NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

  // Issue order: the prologue takes A of steps 0 .. AD-1 and B of steps
  // 0 .. DEPTH-1 (step q's A before its B); step s then issues A of step
  // s + AD and B of step s + DEPTH, A first, also past the last step
  // (clamped addresses, zero scales, stages never read).  LDS DMA is never
  // dropped, so with B through LDS the count of loads issued after A of
  // step t is the same at every step, and so it is inside the main loop,
  // where every register load has a consumer (the next iteration).  In the
  // steps after the loop a B load into registers for a step past the last
  // one has none, and the compiler may drop it: there the waits count only
  // the B loads of real steps (t + j < KTs), never less strict than the
  // schedule needs.
  constexpr int kNA = C::kALoads, kNBl = C::kBLoads, AD = C::kADist, NSA = C::kAStages;
  static_assert(kNBl + (DEPTH - 1) * (kNA + kNBl) <= 63 && 2 * kNBl <= 63, "vmcnt range");
  auto wait_a = [&](int t, auto tail) __attribute__((always_inline)) {
    if constexpr (C::kBLds) {
      // all of step t (A and B): the groups of steps t+1 .. t+DEPTH-1 may remain
      vm_wait<(DEPTH - 1) * (kNA + kNBl)>();
    } else if constexpr (!decltype(tail)::value) {
      if constexpr (AD == DEPTH) vm_wait<kNBl + (DEPTH - 1) * (kNA + kNBl)>();
      else if (t == 0) vm_wait<2 * kNBl>();
      else vm_wait<kNBl>();
    } else if constexpr (AD == DEPTH) {
      // after A(t): B(t), then A of steps t+1 .. t+DEPTH-1 and the B of
      // those that are real steps
      const int live = min(max(KTs - 1 - t, 0), DEPTH - 1);
      vm_wait_live<kNBl + (DEPTH - 1) * kNA, kNBl>(live, std::make_integer_sequence<int, DEPTH>{});
    } else {
      // AD = 1, DEPTH = 2: after A(0): B(0), B(1); after A(t), t >= 1
      // (issued by step t-1): B(t+1); B(1), B(t+1) only if a real step
      const int live = t + 1 < KTs ? 1 : 0;
      if (t == 0) vm_wait_live<kNBl, kNBl>(live, std::make_integer_sequence<int, 2>{});
      else vm_wait_live<0, kNBl>(live, std::make_integer_sequence<int, 2>{});
    }
  };
  auto a_stage = [&](auto slot, int t) __attribute__((always_inline)) {
    if constexpr (NSA == NS) return static_cast<int>(decltype(slot)::value);
    else return t & 1;
  };
  // Lane byte offsets of the A fragments of substep ks inside a stage (row
  // a*32 + l%32 adds a * 4 KiB): logical chunk 4(ks/2) + 2(l/32) + ks%2 at
  // its swizzled position.
  int a_off[kBK / 16];
#pragma unroll
  for (int ks = 0; ks < kBK / 16; ++ks) {
    const int cl = ((ks >> 1) << 2) | ((lane >> 5) << 1) | (ks & 1);
    a_off[ks] = (lane & 31) * (2 * kBK) + 16 * (cl ^ ((lane >> 1) & 7));
  }

  // One K step t: register slot / LDS stage sl = t % (DEPTH + 1) holds step
  // t's operands, the slots of steps t+1 .. t+DEPTH-1 are in flight, and the
  // slot of step t-1 is refilled with step t+DEPTH once every wavefront of
  // the slice is past step t-1 (the barrier at the top of the step).
  auto step = [&](auto slot, int t, auto tail) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot)::value;
    using Refill = std::integral_constant<int, (sl + DEPTH) % NS>;
    wait_a(t, tail);
    slice_sync();
    // [matrix][column half][dword]: substep ks takes dword ks (Q4) or
    // dwords 2ks, 2ks+1 (Q8).
    constexpr int DW = C::kDwords;
    uint32_t bd[NB][2][DW];
    half2v sc[NB][2][2];                                   // [matrix][chunk][column half]
    const char* breg = b_region(sl);
#pragma unroll
    for (int j = 0; j < (C::kFloat ? 0 : NB); ++j)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bool ok = scale_ok(t, c);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          if constexpr (PL) {
            uint32_t w[LW];
            uint32_t sv;
            const int row = 32 * h + (lane & 31), lh = lane >> 5;
            if constexpr (C::kBLds) {
              const char* ch = breg + j * MB + c * CB;
              if constexpr (FMT == QM_Q5_G32 || FMT == QM_Q6_G32) {
                const u32x2 nb = *reinterpret_cast<const u32x2*>(ch + row * 16 + 8 * lh);
                w[0] = nb.x; w[1] = nb.y;
                w[2] = FMT == QM_Q5_G32 ? *reinterpret_cast<const uint32_t*>(ch + 1024 + row * 4)
                                        : *reinterpret_cast<const uint32_t*>(ch + 1024 + row * 8 + 4 * lh);
              } else {
                w[0] = *reinterpret_cast<const uint32_t*>(ch + row * 8 + 4 * lh);
                if constexpr (FMT == QM_Q3_G32) w[1] = *reinterpret_cast<const uint32_t*>(ch + 512 + row * 4);
              }
              sv = *reinterpret_cast<const uint16_t*>(breg + j * MB + 2 * CB + c * 128 + row * 2);
            } else {
#pragma unroll
              for (int i = 0; i < LW; ++i) w[i] = rw[sl][j][c][h][i];
              sv = rs[sl][j][c][h];
            }
            // Bit planes hold the lane's 16 codes at bits 8h.. and 16 + 8h..
            if constexpr (FMT == QM_Q5_G32) w[2] >>= 8 * lh;
            if constexpr (FMT == QM_Q3_G32) w[1] >>= 8 * lh;
            sv = ok ? sv : 0u;
            const _Float16 f = __builtin_bit_cast(_Float16, static_cast<uint16_t>(sv));
            sc[j][c][h] = half2v{f, f};
#pragma unroll
            for (int i = 0; i < LW; ++i) bd[j][h][LW * c + i] = w[i];
            continue;
          }
          BVec d;
          uint32_t sv;
          if constexpr (C::kBLds) {
            const int row = 32 * h + (lane & 31);
            const int in_chunk = Q8 ? row * 16 + 1024 * (lane >> 5) : row * 16 + 8 * (lane >> 5);
            d = *reinterpret_cast<const BVec*>(breg + j * MB + c * CB + in_chunk);
            sv = *reinterpret_cast<const uint16_t*>(breg + j * MB + 2 * CB + c * 128 + row * 2);
          } else {
            d = rb[sl][j][c][h];
            sv = rs[sl][j][c][h];
          }
          sv = ok ? sv : 0u;
          const _Float16 f = __builtin_bit_cast(_Float16, static_cast<uint16_t>(sv));
          sc[j][c][h] = half2v{f, f};
#pragma unroll
          for (int i = 0; i < DW / 2; ++i) bd[j][h][DW / 2 * c + i] = d[i];
        }
      }
    auto dequant = [&](int j, int h, int ks) __attribute__((always_inline)) {
      const int c = ks >> 1, s = ks & 1;
      if constexpr (C::kFloat) {
        // Past the last K step (or a padded panel) the clamped quarter is
        // replaced by zeros: float weights carry no scale to zero it.
        const u32x4 z = {0u, 0u, 0u, 0u};
        const u32x4 v = scale_ok(t, c) ? rf[C::kFloat ? sl : 0][j][c][h][s] : z;
        if constexpr (FMT == QM_F16) {
          return __builtin_bit_cast(half8v, v);
        } else {
          // bf16 -> fp16: exact for every bf16 in fp16's normal range (8
          // significant bits fit in 11); smaller ones round to fp16 subnormals.
          half8v o;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            o[2 * i] = static_cast<_Float16>(__uint_as_float(v[i] << 16));
            o[2 * i + 1] = static_cast<_Float16>(__uint_as_float(v[i] & 0xFFFF0000u));
          }
          return o;
        }
      } else if constexpr (Q8) return dequant_q8(bd[j][h][2 * ks], bd[j][h][2 * ks + 1], sc[j][c][h], dq);
      else if constexpr (FMT == QM_Q5_G32 || FMT == QM_Q6_G32)
        return dequant_nib_hi<FMT>(bd[j][h][LW * c + s], bd[j][h][LW * c + 2], s, sc[j][c][h], dq);
      else if constexpr (FMT == QM_Q2_G32 || FMT == QM_Q3_G32)
        return dequant_crumb<FMT>(bd[j][h][LW * c], FMT == QM_Q3_G32 ? bd[j][h][LW * c + LW - 1] : 0u, s,
                                  sc[j][c][h], dq);
      else return dequant_dword(bd[j][h][ks], sc[j][c][h], dq);
    };
    load_a(a_stage(Refill{}, t + AD), t + AD);             // A, AD steps ahead
    __builtin_amdgcn_sched_barrier(0);
    load_b(Refill{}, t + DEPTH);                           // B, DEPTH steps ahead
    __builtin_amdgcn_sched_barrier(0);                               // keep the loads at the top
    const char* At = a_tile(a_stage(slot, t));
    // Software pipeline over the four 16-deep substeps: the A fragments and
    // the dequantised B fragments of substep ks+1 are produced while the
    // MFMAs of substep ks run.
    half8v af[2][C::kTM];
    half8v bq[2][NB][2];
#pragma unroll
    for (int a = 0; a < C::kTM; ++a) af[0][a] = *reinterpret_cast<const half8v*>(At + a_off[0] + a * 32 * 2 * kBK);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      bq[0][j][0] = dequant(j, 0, 0);
      bq[0][j][1] = dequant(j, 1, 0);
    }
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int cur = ks & 1, nxt = cur ^ 1;
      if (ks + 1 < kBK / 16) {
#pragma unroll
        for (int a = 0; a < C::kTM; ++a)
          af[nxt][a] = *reinterpret_cast<const half8v*>(At + a_off[ks + 1] + a * 32 * 2 * kBK);
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          bq[nxt][j][0] = dequant(j, 0, ks + 1);
          bq[nxt][j][1] = dequant(j, 1, ks + 1);
        }
      }
#pragma unroll
      for (int j = 0; j < NB; ++j) {
#pragma unroll
        for (int a = 0; a < C::kTM; ++a) {
          acc[a][2 * j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[cur][a], bq[cur][j][0], acc[a][2 * j], 0, 0, 0);
          acc[a][2 * j + 1] =
              __builtin_amdgcn_mfma_f32_32x32x16_f16(af[cur][a], bq[cur][j][1], acc[a][2 * j + 1], 0, 0, 0);
        }
      }
    }
  };

  // The kMoeDown row table (and any other LDS written above) is complete and
  // visible before the first DMA is issued (no DMA in flight: the fence
  // costs nothing here).
  if constexpr (MODE == QgMode::kMoeDown) __syncthreads();
  [&]<int... I>(std::integer_sequence<int, I...>) __attribute__((always_inline)) {
    ((I < AD ? load_a(I, I) : void(),
      __builtin_amdgcn_sched_barrier(0),
      load_b(std::integral_constant<int, I>{}, I),
      __builtin_amdgcn_sched_barrier(0)), ...);
  }(std::make_integer_sequence<int, DEPTH>{});
  using Slots = std::make_integer_sequence<int, NS>;
  int t = 0;
  for (; t + NS <= KTs; t += NS) {
    [&]<int... I>(std::integer_sequence<int, I...>) __attribute__((always_inline)) {
      (step(std::integral_constant<int, I>{}, t + I, std::false_type{}), ...);
    }(Slots{});
  }
  [&]<int... I>(std::integer_sequence<int, I...>) __attribute__((always_inline)) {
    ((t + I < KTs ? step(std::integral_constant<int, I>{}, t + I, std::true_type{}) : void()), ...);
  }(Slots{});
  // No LDS DMA may still be in flight when the LDS is reused or the
  // workgroup ends (the prefetches past the last step included).
  vm_wait<0>();

  if constexpr (WK > 1) {
    // Partial sums of slices 1..WK-1 go through LDS; slice 0 adds them in order.
    // The buffer overlaps the A tiles, which slices no longer synchronise on
    // per K step: wait until every slice is done with them.
    __syncthreads();
    float* red = reinterpret_cast<float*>(lds);
    constexpr int per_wave = C::kTM * 2 * NB * 16 * 64;
    if (wk > 0) {
      float* dst = red + ((wk - 1) * WN + wn) * per_wave;
#pragma unroll
      for (int a = 0; a < C::kTM; ++a)
#pragma unroll
        for (int b = 0; b < 2 * NB; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((a * 2 * NB + b) * 16 + r) * 64 + lane] = acc[a][b][r];
    }
    __syncthreads();
    if (wk > 0) return;
#pragma unroll 1
    for (int j = 1; j < WK; ++j) {
      const float* src = red + ((j - 1) * WN + wn) * per_wave;
#pragma unroll
      for (int a = 0; a < C::kTM; ++a)
#pragma unroll
        for (int b = 0; b < 2 * NB; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[a][b][r] += src[((a * 2 * NB + b) * 16 + r) * 64 + lane];
    }
  }

  // Epilogue: lane l, register r of a 32x32 tile holds
  // row 8*(r/4) + 4*(l/32) + r%4, column l%32.
#pragma unroll
  for (int a = 0; a < C::kTM; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int64_t col = n_wave + 32 * b + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int lr = a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (lr >= rows || col >= mN) continue;
        if constexpr (MODE == QgMode::kDense) {
          // Y is not read again by this kernel: stream it past the caches.
          __builtin_nontemporal_store(acc[a][b][r], my + (row0 + lr) * mN + col);
        } else if constexpr (MODE == QgMode::kMoeGateUp) {
          const float g = acc[a][b][r];
          const float u = acc[a][2 + b][r];
          const float hv = g / (1.0f + expf(-g)) * u;
          p.h[(row0 + lr) * N + col] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(hv));
        } else {
          p.yp[row_asg[lr] * N + col] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(row_w[lr] * acc[a][b][r]));
        }
      }
    }
}

}  // namespace qg

// Two workgroups per CU (up to 256 VGPRs per lane) for up to 4 wavefronts
// per workgroup, one beyond.  NT: weights and scales are read with
// nontemporal loads (for weights each workgroup streams once and no other
// workgroup re-reads soon).  FMT: any of the eight weight formats.
template <int BM, int WN, int WK, QgMode MODE, int DEPTH = 2, bool NT = false, int FMT = QM_Q4_G32>
__global__ __launch_bounds__(WN * WK * 64, WN * WK <= 4 ? 2 : 1) void qgemm_kernel(QgemmArgs p) {
  qg::qgemm_body<BM, WN, WK, MODE, DEPTH, NT, FMT>(p);
}

}  // namespace qm
