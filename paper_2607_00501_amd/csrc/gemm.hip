// Prefill GEMM  Y[m][n] = sum_k X[m][k] * w'[n][k]  with Q4 weights
// dequantised inside the kernel and fp16 MFMA (BaseRT Sec. 3.4: tiled GEMM
// for the prompt, tile geometry chosen by sequence-length regime; Sec. 3.3:
// dequantisation lives inside the GEMM, weights are never materialised).
// The kernel itself is the shared Q4 MFMA core in qgemm.h (dense mode);
// this file holds the per-chip tile plan and the launch.
#include <cstdio>
#include <cstdlib>

#include "qgemm.h"

namespace qm {
namespace {

template <int BM, int WN, int WK>
hipError_t launch_tile(const QgemmArgs& a, hipStream_t st) {
  const int64_t panels = a.gpanel[a.gcount];
  const dim3 grid(static_cast<unsigned>((panels + WN - 1) / WN), static_cast<unsigned>((a.M + BM - 1) / BM));
  hipLaunchKernelGGL((qgemm_kernel<BM, WN, WK, QgMode::kDense>), grid, dim3(WN * WK * 64), 0, st, a);
  return hipGetLastError();
}

}  // namespace

// Per-chip tile choice by M regime (Sec. 3.4: tiles tuned to sequence
// length), fitted to a per-shape sweep on MI355X (256 CUs): the 128 x 256
// tile when it gives at least two workgroups per CU, else the 64 x 256 tile
// when it gives one per CU; else one 64-column panel per K slice with
// split-K over as many one-wavefront slices as keep >= 8 K steps each (at
// most 8), in 64-row tiles if that gives 8 wavefronts per CU, else 32-row
// tiles.
GemmPlan gemm_plan(int64_t m, int64_t n, int64_t k, int cu_count) {
  // Tuning sweeps only: QM_GEMM_PLAN="bm,wn,wk" forces the plan.
  static const GemmPlan forced = [] {
    GemmPlan f{0, 0, 0};
    if (const char* e = std::getenv("QM_GEMM_PLAN")) std::sscanf(e, "%d,%d,%d", &f.bm, &f.wn, &f.wk);
    return f;
  }();
  if ((forced.bm == 32 || forced.bm == 64 || forced.bm == 128) && (forced.wn == 1 || forced.wn == 2 || forced.wn == 4) &&
      (forced.wk == 1 || forced.wk == 2 || forced.wk == 4 || forced.wk == 8)) {
    GemmPlan f = forced;
    if (f.wk > 1 || f.bm == 32) { f.wn = 1; if (f.bm == 128) f.bm = 64; }
    return f;
  }
  auto blocks = [&](int bm, int wn) { return ((n + 64 * wn - 1) / (64 * wn)) * ((m + bm - 1) / bm); };
  if (blocks(128, 4) >= 2 * cu_count) return GemmPlan{128, 4, 1};
  if (blocks(64, 4) >= cu_count) return GemmPlan{64, 4, 1};
  const int64_t kt = (k / kGroup + 1) / 2;
  int wk = 1;
  while (wk < 8 && kt / (2 * wk) >= 8) wk *= 2;
  if (blocks(64, 1) * wk >= 8 * static_cast<int64_t>(cu_count)) return GemmPlan{64, 1, wk};
  return GemmPlan{32, 1, wk};
}

const char* gemm_tile_name(int64_t m, int64_t n) {
  static thread_local char buf[64];
  const GemmPlan p = gemm_plan(m, n, 2048, 256);
  std::snprintf(buf, sizeof(buf), "BM%d x %d, %d-way split-K", p.bm, 64 * p.wn, p.wk);
  return buf;
}

namespace {

hipError_t launch_args(const QgemmArgs& a, int cu_count, hipStream_t st) {
  const int64_t panels = a.gpanel[a.gcount];
  if (panels == 0) return hipSuccess;
  const GemmPlan p = gemm_plan(a.M, panels * kPanel, a.K, cu_count);
  if (p.wn == 4) {
    if (p.bm == 128) return launch_tile<128, 4, 1>(a, st);
    return launch_tile<64, 4, 1>(a, st);
  }
  if (p.wn == 2) return launch_tile<64, 2, 1>(a, st);
  if (p.bm == 64) {
    switch (p.wk) {
      case 1: return launch_tile<64, 1, 1>(a, st);
      case 2: return launch_tile<64, 1, 2>(a, st);
      case 4: return launch_tile<64, 1, 4>(a, st);
      default: return launch_tile<64, 1, 8>(a, st);
    }
  }
  switch (p.wk) {
    case 1: return launch_tile<32, 1, 1>(a, st);
    case 2: return launch_tile<32, 1, 2>(a, st);
    case 4: return launch_tile<32, 1, 4>(a, st);
    default: return launch_tile<32, 1, 8>(a, st);
  }
}

}  // namespace

hipError_t launch_gemm(const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y, int64_t m,
                       int64_t n, int64_t k, int cu_count, hipStream_t st) {
  const uint8_t* qs[1] = {q};
  const uint16_t* ss[1] = {s};
  float* ys[1] = {y};
  const int64_t ns[1] = {n};
  return launch_gemm_group(1, qs, ss, ys, ns, x, m, k, cu_count, st);
}

hipError_t launch_gemm_group(int count, const uint8_t* const* q, const uint16_t* const* s, float* const* y,
                             const int64_t* n, const uint16_t* x, int64_t m, int64_t k, int cu_count,
                             hipStream_t st) {
  QgemmArgs a{};
  a.a = x; a.M = m; a.K = k;
  a.q = q[0]; a.s = s[0]; a.y = y[0]; a.N = n[0];
  a.gcount = count;
  a.gpanel[0] = 0;
  for (int i = 0; i < count; ++i) {
    a.gq[i] = q[i]; a.gs[i] = s[i]; a.gy[i] = y[i]; a.gn[i] = n[i];
    a.gpanel[i + 1] = a.gpanel[i] + static_cast<int32_t>(padded_rows(n[i]) / kPanel);
  }
  return launch_args(a, cu_count, st);
}

}  // namespace qm
