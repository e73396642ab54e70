// Prefill GEMM  Y[m][n] = sum_k X[m][k] * w'[n][k]  with Q4 weights
// dequantised inside the kernel and fp16 MFMA (BaseRT Sec. 3.4: tiled GEMM
// for the prompt, tile geometry chosen by sequence-length regime; Sec. 3.3:
// dequantisation lives inside the GEMM, weights are never materialised).
//
// Mapping on gfx950 (64-lane wavefronts, v_mfma_f32_32x32x16_f16):
//  * a workgroup has WN x WK wavefronts; wavefront (wn, wk) owns the BM x 64
//    output block whose 64 columns are one device-layout panel, over the
//    wk-th slice of the K steps (WK > 1 is split-K inside the workgroup for
//    long-K, small-grid shapes; the partial sums meet in LDS in a fixed
//    order).  One 64-deep K step of its weights is two 1 KiB contiguous
//    chunk rows: one dwordx4 per lane per chunk, fully coalesced;
//  * the weights never pass through LDS: each wavefront dequantises its own
//    B fragments in registers.  One v_permlane32_swap per dword pair moves
//    the codes of panel rows 32..63 / 0..31 into the MFMA B-operand lane
//    layout (lane l holds 8 consecutive k of column l%32); v_and_or_b32 +
//    v_pk_add_f16 + v_pk_mul_f16 then give fp16_RNE(s*q) exactly.  The
//    dequantisation of each 16-k substep is interleaved with the MFMAs of
//    the previous one;
//  * the activation tile of each K slice (BM x 64 fp16) is double-buffered
//    in LDS (one barrier per K step) and shared by the WN wavefronts of the
//    slice; A fragments of the next substep are read while the current
//    MFMAs run;
//  * global loads run two K steps ahead of the MFMAs.  Out-of-range rows,
//    columns and K steps read clamped (valid) addresses with their scales
//    forced to zero, so the loads carry no branches.
#include "qm_internal.h"

#include <cstdio>
#include <cstdlib>
#include <type_traits>

namespace qm {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBK = 64;                 // K per step (two quantisation groups)
constexpr int kRow = kBK + 8;           // LDS row stride in halves (16-byte pad)

__device__ inline uint32_t and_or_v(uint32_t a, uint32_t mask_v, uint32_t or_s) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(mask_v), "s"(or_s));
  return r;
}

// 8 offset-binary nibbles of one device-layout dword (k order 0,2,4,6 |
// 1,3,5,7) -> 8 fp16 fp16_RNE(s*q) in natural k order.
__device__ inline half8v dequant_dword(uint32_t d, half2v s2) {
  const half2v bias = {(_Float16)1032.0f, (_Float16)1032.0f};
  const uint32_t m0 = 0x000F000Fu, magic = 0x64006400u;
  half8v out;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const half2v q = __builtin_bit_cast(half2v, and_or_v(d >> (4 * i), m0, magic)) - bias;
    const half2v v = q * s2;
    out[2 * i] = v[0];
    out[2 * i + 1] = v[1];
  }
  return out;
}

template <int BM, int WN, int WK>
struct GemmCfg {
  static constexpr int kThreads = WN * WK * 64;
  static constexpr int kSliceThreads = WN * 64;
  static constexpr int kTM = BM / 32;
  static constexpr int kALoads = BM * (kBK / 8) / kSliceThreads;
  static constexpr int kStage = BM * kRow;                        // halves per A stage
  static_assert(kALoads >= 1 && BM * (kBK / 8) % kSliceThreads == 0, "A tile split");
  static_assert(WK == 1 || (WK - 1) * WN * BM * 64 * 4 <= 2 * WK * kStage * 2, "reduction fits in LDS");
};

template <int BM, int WN, int WK>
__global__ __launch_bounds__(WN * WK * 64, 2) void gemm_q4_kernel(const uint8_t* __restrict__ q,
                                                               const uint16_t* __restrict__ s,
                                                               const uint16_t* __restrict__ x,
                                                               float* __restrict__ y, int64_t M,
                                                               int64_t N, int64_t K) {
  using C = GemmCfg<BM, WN, WK>;
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * WK * C::kStage];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wk = wave / WN, wn = wave % WN;
  const int stid = tid - wk * C::kSliceThreads;          // thread index inside the K slice
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * BM;
  const int64_t n_wave = static_cast<int64_t>(blockIdx.x) * (64 * WN) + 64 * wn;
  const int G = static_cast<int>(K / kGroup);
  const int KT = (G + 1) / 2;
  const int KTs = (KT + WK - 1) / WK;                      // K steps per slice
  const int kt0 = wk * KTs;
  const int64_t npad = padded_rows(N);
  const bool cols_ok = n_wave < npad;

  // A: this thread's rows/cols of the slice's BM x 64 tile (rows clamped).
  const uint16_t* a_src[C::kALoads];
  int a_lds[C::kALoads], a_col[C::kALoads];
#pragma unroll
  for (int i = 0; i < C::kALoads; ++i) {
    const int idx = stid + i * C::kSliceThreads;
    const int row = idx >> 3;
    a_col[i] = (idx & 7) * 8;
    a_lds[i] = row * kRow + a_col[i];
    const int64_t r = m0 + row < M ? m0 + row : M - 1;
    a_src[i] = x + r * K;
  }
  // B: lane l streams row l of the wavefront's panel (clamped to a real panel).
  const int64_t panel = (cols_ok ? n_wave : npad - kPanel) / kPanel;
  const uint8_t* b_q = q + (panel * G * kPanel + lane) * 16;
  const uint16_t* b_s = s + panel * G * kPanel + lane;

  // Two register sets of raw step operands, always indexed by constants.
  u32x4 ra[2][C::kALoads];
  u32x4 rb[2][2];
  uint32_t rs[2][2];
  auto load = [&](auto slot, int step) __attribute__((always_inline)) {
    constexpr int p = decltype(slot)::value;
    const int kt = kt0 + step;
#pragma unroll
    for (int i = 0; i < C::kALoads; ++i) {
      const int k = min(kt * kBK + a_col[i], static_cast<int>(K) - 8);
      ra[p][i] = *reinterpret_cast<const u32x4*>(a_src[i] + k);
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int g = 2 * kt + c;
      const int gc = min(g, G - 1);
      rb[p][c] = *reinterpret_cast<const u32x4*>(b_q + static_cast<int64_t>(gc) * kPanel * 16);
      const uint32_t sv = b_s[static_cast<int64_t>(gc) * kPanel];
      rs[p][c] = (cols_ok && g < G && step < KTs && kt < KT) ? sv : 0u;
    }
  };
  auto store_a = [&](auto slot, int buf) __attribute__((always_inline)) {
    constexpr int p = decltype(slot)::value;
    uint16_t* dst = lds + (buf * WK + wk) * C::kStage;
#pragma unroll
    for (int i = 0; i < C::kALoads; ++i) *reinterpret_cast<u32x4*>(dst + a_lds[i]) = ra[p][i];
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;

  float16v acc[C::kTM][2];
#pragma unroll
  for (int a = 0; a < C::kTM; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

  // One K step t: register slot p holds step t's raw operands (its A tile is
  // already in LDS buffer t&1), slot 1-p step t+1's.  The B codes of slot p
  // move to registers in MFMA layout, then slot p is refilled with step t+2;
  // step t+1's A tile goes to the other LDS buffer after the MFMAs.
  auto step = [&](auto slot, int t) __attribute__((always_inline)) {
    constexpr int p = decltype(slot)::value;          // slot p: step t, slot 1-p: step t+1
    using Next = std::integral_constant<int, 1 - p>;
    const int buf = t & 1;
    uint32_t bd[2][4];                                     // [column half][substep]
    half2v sc[2][2];                                       // [chunk][column half]
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const auto sw = __builtin_amdgcn_permlane32_swap(rs[p][c], rs[p][c], false, false);
      const _Float16 lo = __builtin_bit_cast(_Float16, static_cast<uint16_t>(sw[0]));
      const _Float16 hi = __builtin_bit_cast(_Float16, static_cast<uint16_t>(sw[1]));
      sc[c][0] = half2v{lo, lo};
      sc[c][1] = half2v{hi, hi};
      const uint32_t d[4] = {rb[p][c][0], rb[p][c][1], rb[p][c][2], rb[p][c][3]};
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const auto p = __builtin_amdgcn_permlane32_swap(d[2 * i], d[2 * i + 1], false, false);
        bd[0][2 * c + i] = p[0];                           // panel rows 0..31
        bd[1][2 * c + i] = p[1];                           // panel rows 32..63
      }
    }
    load(slot, t + 2);                                     // two steps ahead
    __builtin_amdgcn_sched_barrier(0);                     // keep the loads at the top
    const uint16_t* At = lds + (buf * WK + wk) * C::kStage + (lane & 31) * kRow + 8 * (lane >> 5);
    half8v af[2][C::kTM];
#pragma unroll
    for (int a = 0; a < C::kTM; ++a) af[0][a] = *reinterpret_cast<const half8v*>(At + a * 32 * kRow);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      if (ks + 1 < kBK / 16) {
#pragma unroll
        for (int a = 0; a < C::kTM; ++a)
          af[(ks + 1) & 1][a] = *reinterpret_cast<const half8v*>(At + a * 32 * kRow + (ks + 1) * 16);
      }
      const half8v b0 = dequant_dword(bd[0][ks], sc[ks >> 1][0]);
      const half8v b1 = dequant_dword(bd[1][ks], sc[ks >> 1][1]);
#pragma unroll
      for (int a = 0; a < C::kTM; ++a) {
        acc[a][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[ks & 1][a], b0, acc[a][0], 0, 0, 0);
        acc[a][1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[ks & 1][a], b1, acc[a][1], 0, 0, 0);
      }
    }
    if (t + 1 < KTs) store_a(Next{}, buf ^ 1);
    __syncthreads();
  };

  load(S0{}, 0);
  load(S1{}, 1);
  store_a(S0{}, 0);
  __syncthreads();
  int t = 0;
  for (; t + 2 <= KTs; t += 2) {
    step(S0{}, t);
    step(S1{}, t + 1);
  }
  if (t < KTs) step(S0{}, t);

  if (WK > 1) {
    // Partial sums of slices 1..WK-1 go through LDS; slice 0 adds them in order.
    float* red = reinterpret_cast<float*>(lds);
    if (wk > 0) {
      float* dst = red + ((wk - 1) * WN + wn) * (C::kTM * 2 * 16 * 64);
#pragma unroll
      for (int a = 0; a < C::kTM; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[((a * 2 + b) * 16 + r) * 64 + lane] = acc[a][b][r];
    }
    __syncthreads();
    if (wk > 0) return;
    for (int j = 1; j < WK; ++j) {
      const float* src = red + ((j - 1) * WN + wn) * (C::kTM * 2 * 16 * 64);
#pragma unroll
      for (int a = 0; a < C::kTM; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[a][b][r] += src[((a * 2 + b) * 16 + r) * 64 + lane];
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
        const int64_t row = m0 + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < M && col < N) y[row * N + col] = acc[a][b][r];
      }
    }
}

template <int BM, int WN, int WK>
hipError_t launch_tile(const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y, int64_t m,
                       int64_t n, int64_t k, hipStream_t st) {
  const dim3 grid(static_cast<unsigned>((n + 64 * WN - 1) / (64 * WN)),
                  static_cast<unsigned>((m + BM - 1) / BM));
  hipLaunchKernelGGL((gemm_q4_kernel<BM, WN, WK>), grid, dim3(WN * WK * 64), 0, st, q, s, x, y, m, n, k);
  return hipGetLastError();
}

}  // namespace

// Per-chip tile choice by M regime (Sec. 3.4: tiles tuned to sequence
// length), fitted to a per-shape sweep on MI355X (256 CUs): the 128 x 256
// tile when it gives at least two workgroups per CU, else the 64 x 256 tile
// when it gives one per CU, else one panel per workgroup with split-K over
// up to 4 wavefronts (at least 8 K steps per slice).
GemmPlan gemm_plan(int64_t m, int64_t n, int64_t k, int cu_count) {
  // Tuning sweeps only: QM_GEMM_PLAN="bm,wn,wk" forces the plan.
  static const GemmPlan forced = [] {
    GemmPlan f{0, 0, 0};
    if (const char* e = std::getenv("QM_GEMM_PLAN")) std::sscanf(e, "%d,%d,%d", &f.bm, &f.wn, &f.wk);
    return f;
  }();
  if ((forced.bm == 64 || forced.bm == 128) && (forced.wn == 1 || forced.wn == 2 || forced.wn == 4) &&
      (forced.wk == 1 || forced.wk == 2 || forced.wk == 4)) {
    GemmPlan f = forced;
    if (f.wk > 1) { f.bm = 64; f.wn = 1; }
    return f;
  }
  auto blocks = [&](int bm, int wn) { return ((n + 64 * wn - 1) / (64 * wn)) * ((m + bm - 1) / bm); };
  if (blocks(128, 4) >= 2 * cu_count) return GemmPlan{128, 4, 1};
  if (blocks(64, 4) >= cu_count) return GemmPlan{64, 4, 1};
  GemmPlan p{64, 1, 1};
  const int64_t kt = (k / kGroup + 1) / 2;
  while (p.wk < 4 && blocks(64, 1) * p.wk < 4 * cu_count && kt / (2 * p.wk) >= 8) p.wk *= 2;
  return p;
}

const char* gemm_tile_name(int64_t m, int64_t n) {
  static thread_local char buf[64];
  const GemmPlan p = gemm_plan(m, n, 2048, 256);
  std::snprintf(buf, sizeof(buf), "BM%d x %d, %d-way split-K", p.bm, 64 * p.wn, p.wk);
  return buf;
}

hipError_t launch_gemm(const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y, int64_t m,
                       int64_t n, int64_t k, int cu_count, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const GemmPlan p = gemm_plan(m, n, k, cu_count);
  if (p.wk == 1) {
    if (p.bm == 128) {
      if (p.wn == 4) return launch_tile<128, 4, 1>(q, s, x, y, m, n, k, st);
      return launch_tile<128, 2, 1>(q, s, x, y, m, n, k, st);
    }
    if (p.wn == 4) return launch_tile<64, 4, 1>(q, s, x, y, m, n, k, st);
    if (p.wn == 2) return launch_tile<64, 2, 1>(q, s, x, y, m, n, k, st);
    return launch_tile<64, 1, 1>(q, s, x, y, m, n, k, st);
  }
  if (p.wk == 2) return launch_tile<64, 1, 2>(q, s, x, y, m, n, k, st);
  return launch_tile<64, 1, 4>(q, s, x, y, m, n, k, st);
}

}  // namespace qm
