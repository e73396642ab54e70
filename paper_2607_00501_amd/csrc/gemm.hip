// Prefill GEMM  Y[m][n] = sum_k X[m][k] * w'[n][k]  with Q4 weights
// dequantised into LDS and fp16 MFMA (BaseRT Sec. 3.4: tiled GEMM for the
// prompt, tile geometry chosen by sequence-length regime; Sec. 3.3: the
// dequantisation lives inside the GEMM kernel).
#include "mfma_tile.h"

namespace qm {
namespace {

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64) void gemm_q4_kernel(const uint8_t* __restrict__ q,
                                                               const uint16_t* __restrict__ s,
                                                               const uint16_t* __restrict__ x,
                                                               float* __restrict__ y, int64_t M,
                                                               int64_t N, int64_t K) {
  using T = MfmaTile<BM, BN, WM, WN, false>;
  __shared__ __attribute__((aligned(16))) uint16_t lds[T::kLdsBytes / 2];
  const int64_t n0 = static_cast<int64_t>(blockIdx.x) * BN;
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * BM;
  const int64_t G = K / kGroup;
  const int64_t npad = padded_rows(N);

  const uint16_t* a_rows[T::kALoads];
#pragma unroll
  for (int i = 0; i < T::kALoads; ++i) {
    const int64_t row = m0 + T::a_row(i);
    a_rows[i] = row < M ? x + row * K : nullptr;
  }
  const uint8_t* b_q[T::kBLoads];
  const uint16_t* b_s[T::kBLoads];
#pragma unroll
  for (int i = 0; i < T::kBLoads; ++i) {
    const int64_t n = n0 + T::b_row(i);
    b_q[i] = n < npad ? q4_row_chunk0(q, n, G) : nullptr;
    b_s[i] = n < npad ? q4_row_scale0(s, n, G) : nullptr;
  }
  float16v acc[T::kTM][T::kTN];
  T::run(a_rows, b_q, b_s, static_cast<int>(K), lds, acc);

#pragma unroll
  for (int a = 0; a < T::kTM; ++a)
#pragma unroll
    for (int b = 0; b < T::kTN; ++b) {
      const int64_t col = n0 + T::out_col(b);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + T::out_row(a, r);
        if (row < M && col < N) y[row * N + col] = acc[a][b][r];
      }
    }
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_tile(const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y, int64_t m,
                       int64_t n, int64_t k, hipStream_t st) {
  const dim3 grid(static_cast<unsigned>((n + BN - 1) / BN), static_cast<unsigned>((m + BM - 1) / BM));
  hipLaunchKernelGGL((gemm_q4_kernel<BM, BN, WM, WN>), grid, dim3(WM * WN * 64), 0, st, q, s, x, y, m, n,
                     k);
  return hipGetLastError();
}

}  // namespace

// Per-chip tile choice by M regime.
const char* gemm_tile_name(int64_t m, int64_t n) {
  (void)n;
  return m <= 128 ? "64x128(2x2 waves)" : "128x128(2x2 waves)";
}

hipError_t launch_gemm(const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y, int64_t m,
                       int64_t n, int64_t k, int cu_count, hipStream_t st) {
  (void)cu_count;
  if (n == 0) return hipSuccess;
  if (m <= 128) return launch_tile<64, 128, 2, 2>(q, s, x, y, m, n, k, st);
  return launch_tile<128, 128, 2, 2>(q, s, x, y, m, n, k, st);
}

}  // namespace qm
