// Prefill GEMM  Y[m][n] = sum_k X[m][k] * w'[n][k]  with Q2 .. Q8 weights
// dequantised inside the kernel, or F16 / BF16 weights taken as they are
// (BF16 converted to fp16 in registers), and fp16 MFMA (BaseRT Sec. 3.4: tiled GEMM
// for the prompt, tile geometry chosen by sequence-length regime; Sec. 3.3:
// dequantisation lives inside the GEMM, weights are never materialised).
// The kernel itself is the shared MFMA core in qgemm.h (dense mode);
// this file holds the per-chip tile plan and the launch.
#include <cstdio>
#include <cstdlib>

#include "qgemm.h"

namespace qm {
namespace {

template <int BM, int WN, int WK, int FMT>
hipError_t launch_tile(const QgemmArgs& a, hipStream_t st) {
  const int64_t panels = a.gpanel[a.gcount];
  const dim3 grid(static_cast<unsigned>((panels + WN - 1) / WN), static_cast<unsigned>((a.M + BM - 1) / BM));
  hipLaunchKernelGGL((qgemm_kernel<BM, WN, WK, QgMode::kDense, 2, false, FMT>), grid, dim3(WN * WK * 64), 0, st,
                     a);
  return hipGetLastError();
}

}  // namespace

// Per-chip tile choice by M regime (Sec. 3.4: tiles tuned to sequence
// length), fitted to per-shape sweeps on MI355X (256 CUs) over the
// Llama-3.2-1B, Llama-3.2-3B and Qwen3-0.6B shapes and their grouped widths
// at M = 128, 512, 2048 (K steps of 64):
//  * 128 x 256 tiles when they give at least 3/4 workgroup per CU;
//  * else 64 x 256 tiles when they give at least 3/4 per CU;
//  * else 64 x 128 tiles with 2-way split-K when those give at least 3/4
//    workgroup per CU and K has >= 16 steps;
//  * else one 64-column panel per K slice with split-K over as many
//    one-wavefront slices as keep >= 8 K steps each (>= 4 when K has fewer
//    than 32 steps; at most 8 slices), in 64-row tiles if that gives 4
//    wavefronts per CU, else 32-row tiles.
// (The K < 2048 thresholds took the Qwen3-0.6B shapes 1024 -> 4096 / 6144
// from 301 / 396 to 373 / 443 TFLOP/s at M = 512 and from 142 / 160 to
// 164 / 178 at M = 128; no plan of the other models changed.)
// The other formats use the same plan.  Where their weight stages do not fit
// in LDS beside the A stages (Q8, Q5, Q6 at 128 x 256) the tile keeps the
// weights in registers; for Q8 that still beats 64 x 256 tiles by 10-20%
// where the rule picks it.  F16 / BF16 weights always go through registers:
// each lane's 16-byte quarters are already MFMA B fragments.
GemmPlan gemm_plan(int64_t m, int64_t n, int64_t k, int cu_count) {
  // Tuning sweeps only: QM_GEMM_PLAN="bm,wn,wk" forces the plan (one of the
  // instantiated tiles, see launch_args).
  static const GemmPlan forced = [] {
    GemmPlan f{0, 0, 0};
    if (const char* e = tuning_override("QM_GEMM_PLAN")) std::sscanf(e, "%d,%d,%d", &f.bm, &f.wn, &f.wk);
    return f;
  }();
  if (forced.bm != 0 && gemm_plan_instantiated(forced)) return forced;
  auto blocks = [&](int bm, int wn) { return ((n + 64 * wn - 1) / (64 * wn)) * ((m + bm - 1) / bm); };
  const int64_t cu = cu_count;
  const int64_t kt = (k / kGroup + 1) / 2;
  if (4 * blocks(128, 4) >= 3 * cu) return GemmPlan{128, 4, 1};
  if (4 * blocks(64, 4) >= 3 * cu) return GemmPlan{64, 4, 1};
  if (4 * blocks(64, 2) >= 3 * cu && kt >= 16) return GemmPlan{64, 2, 2};
  const int64_t min_steps = kt < 32 ? 4 : 8;
  int wk = 1;
  while (wk < 8 && kt / (2 * wk) >= min_steps) wk *= 2;
  if (blocks(64, 1) * wk >= 4 * cu) return GemmPlan{64, 1, wk};
  return GemmPlan{32, 1, wk};
}

const char* gemm_tile_name(int64_t m, int64_t n) {
  static thread_local char buf[64];
  const GemmPlan p = gemm_plan(m, n, 2048, 256);
  std::snprintf(buf, sizeof(buf), "BM%d x %d, %d-way split-K", p.bm, 64 * p.wn, p.wk);
  return buf;
}

namespace {

// The tiles gemm_plan() can choose (QM_GEMM_PLAN may force any of them).
// Every format instantiates the same tiles.
#define QM_GEMM_TILES(X) \
  X(128, 4, 1) X(64, 4, 1) X(64, 2, 2) \
  X(64, 1, 1) X(64, 1, 2) X(64, 1, 4) X(64, 1, 8) X(32, 1, 1) X(32, 1, 2) X(32, 1, 4) X(32, 1, 8)

hipError_t launch_args(const QgemmArgs& a, int32_t fmt, int cu_count, hipStream_t st) {
  const int64_t panels = a.gpanel[a.gcount];
  if (panels == 0) return hipSuccess;
  const GemmPlan p = gemm_plan(a.M, panels * kPanel, a.K, cu_count);
#define QM_LAUNCH_FMT(F) \
  if (fmt == F) {                                                                            \
    QM_GEMM_TILES(QM_LAUNCH_TILE)                                                            \
    return hipErrorInvalidConfiguration;                                                     \
  }
#define QM_LAUNCH_TILE(BM, WN, WK) \
  if (p.bm == BM && p.wn == WN && p.wk == WK) return launch_tile<BM, WN, WK, F_>(a, st);
  {
    constexpr int F_ = QM_Q4_G32;
    QM_LAUNCH_FMT(QM_Q4_G32)
  }
  {
    constexpr int F_ = QM_Q8_G32;
    QM_LAUNCH_FMT(QM_Q8_G32)
  }
  {
    constexpr int F_ = QM_Q2_G32;
    QM_LAUNCH_FMT(QM_Q2_G32)
  }
  {
    constexpr int F_ = QM_Q3_G32;
    QM_LAUNCH_FMT(QM_Q3_G32)
  }
  {
    constexpr int F_ = QM_Q5_G32;
    QM_LAUNCH_FMT(QM_Q5_G32)
  }
  {
    constexpr int F_ = QM_Q6_G32;
    QM_LAUNCH_FMT(QM_Q6_G32)
  }
  {
    constexpr int F_ = QM_F16;
    QM_LAUNCH_FMT(QM_F16)
  }
  {
    constexpr int F_ = QM_BF16;
    QM_LAUNCH_FMT(QM_BF16)
  }
#undef QM_LAUNCH_TILE
#undef QM_LAUNCH_FMT
  return hipErrorInvalidValue;
}

}  // namespace

bool gemm_plan_instantiated(const GemmPlan& p) {
#define QM_HAS(BM, WN, WK) \
  if (p.bm == BM && p.wn == WN && p.wk == WK) return true;
  QM_GEMM_TILES(QM_HAS)
#undef QM_HAS
  return false;
}

hipError_t launch_gemm(int32_t fmt, const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y, int64_t m,
                       int64_t n, int64_t k, int cu_count, hipStream_t st) {
  const uint8_t* qs[1] = {q};
  const uint16_t* ss[1] = {s};
  float* ys[1] = {y};
  const int64_t ns[1] = {n};
  return launch_gemm_group(fmt, 1, qs, ss, ys, ns, x, m, k, cu_count, st);
}

hipError_t launch_gemm_group(int32_t fmt, int count, const uint8_t* const* q, const uint16_t* const* s,
                             float* const* y, const int64_t* n, const uint16_t* x, int64_t m, int64_t k,
                             int cu_count, hipStream_t st) {
  QgemmArgs a{};
  a.a = x; a.M = m; a.K = k;
  a.q = q[0]; a.s = s[0]; a.y = y[0]; a.N = n[0];
  a.gcount = count;
  a.gpanel[0] = 0;
  for (int i = 0; i < count; ++i) {
    a.gq[i] = q[i]; a.gs[i] = s[i]; a.gy[i] = y[i]; a.gn[i] = n[i];
    a.gpanel[i + 1] = a.gpanel[i] + static_cast<int32_t>(padded_rows(n[i]) / kPanel);
  }
  return launch_args(a, fmt, cu_count, st);
}

}  // namespace qm
