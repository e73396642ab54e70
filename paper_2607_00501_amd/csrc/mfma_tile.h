// Block-tiled fp16 MFMA main loop with Q4 weight tiles dequantised into LDS.
//
// This is the GEMM half of the quantised matmul (BaseRT Sec. 3.3 / Sec. 3.4:
// prefill uses tiled GEMM kernels on the matrix units, with dequantisation
// inside the kernel rather than materialised).  On gfx950 one workgroup of
// WM x WN wavefronts owns a BM x BN output tile:
//   * every K step (BK = 64, two quantisation groups) the activation tile
//     (fp16, BM x 64) is copied global -> registers -> LDS, and the weight
//     tile (BN rows x 2 chunks of the device layout, 1 KiB contiguous per 64
//     rows) is loaded, dequantised once in registers to fp16_RNE(s * q)
//     (v_and_or_b32 -> fp16 1024+u, packed subtract 1032, packed multiply by
//     the fp16 scale: a single rounding of the exact product) and stored to
//     LDS, so each weight is dequantised once per workgroup, not per wave;
//   * each wavefront runs v_mfma_f32_32x32x16_f16 over its (BM/WM) x (BN/WN)
//     sub-tile with fp32 accumulators;
//   * the next K step's global loads are issued before the MFMAs of the
//     current one, so HBM latency overlaps matrix work.
// With DUAL the B tile holds two weight matrices at the same rows (the gate
// and up projections of a SwiGLU expert): rows [0, BN/2) come from the first,
// rows [BN/2, BN) from the second, and each wavefront owns matching column
// blocks of both, so the epilogue sees gate and up values in the same lane.
#pragma once

#include "qm_internal.h"

namespace qm {

constexpr int kBK = 64;          // K per main-loop step (two groups)
constexpr int kLdsPad = 8;       // halves of padding per LDS row
constexpr int kLdsRow = kBK + kLdsPad;

__device__ inline uint32_t tile_and_or(uint32_t a, uint32_t mask_v, uint32_t or_s) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(mask_v), "s"(or_s));
  return r;
}

// Dequantise one 16-byte Q4 device chunk (32 weights, natural k order out)
// into 16 fp16 pairs fp16_RNE(s * q).
__device__ inline void dequant_chunk_f16(const uint4 w, uint16_t sbits, uint32_t out[16]) {
  const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
  const half2v bias = {(_Float16)1032.0f, (_Float16)1032.0f};
  const _Float16 sh = __builtin_bit_cast(_Float16, sbits);
  const half2v s2 = {sh, sh};
  const uint32_t m0 = 0x000F000Fu;
  const uint32_t magic = 0x64006400u;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t h = tile_and_or(wd[j] >> (4 * i), m0, magic);
      const half2v q = __builtin_bit_cast(half2v, h) - bias;   // exact integers
      out[4 * j + i] = __builtin_bit_cast(uint32_t, q * s2);   // one rounding
    }
  }
}

template <int BM, int BN, int WM, int WN, bool DUAL>
struct MfmaTile {
  static constexpr int kThreads = WM * WN * 64;
  static constexpr int kTM = BM / WM / 32;                       // 32x32 tiles per wave (M)
  static constexpr int kTN = BN / WN / 32;                       // 32x32 tiles per wave (N)
  static constexpr int kALoads = BM * (kBK / 8) / kThreads;      // 16-byte A loads per thread
  static constexpr int kBLoads = BN * 2 / kThreads;              // chunk loads per thread
  static constexpr int kBNh = DUAL ? BN / 2 : BN;
  static_assert(BM % (WM * 32) == 0 && BN % (WN * 32) == 0, "wave tile must be 32-aligned");
  static_assert(kALoads >= 1 && BM * (kBK / 8) % kThreads == 0, "A tile must split evenly");
  static_assert(kBLoads >= 1 && BN * 2 % kThreads == 0, "B tile must split evenly");
  static_assert(kBNh % 64 == 0, "B rows per matrix must be whole panels");
  static_assert(!DUAL || (kTN % 2 == 0), "DUAL needs matching gate/up column blocks");
  static constexpr size_t kLdsBytes = static_cast<size_t>(BM + BN) * kLdsRow * 2;

  // Column (within the B tile) of the wave's n-block tn.
  __device__ static int b_col(int wn, int tn) {
    if (!DUAL) return wn * (BN / WN) + tn * 32;
    constexpr int half_tiles = kTN / 2;
    const int base = wn * (kBNh / WN);
    return tn < half_tiles ? base + tn * 32 : kBNh + base + (tn - half_tiles) * 32;
  }

  // Runs the K loop.  a_rows[i]: source row of this thread's i-th A load
  // (nullptr -> zeros); b_q[i]/b_s[i]: first chunk / scale of the thread's
  // i-th B row in its device-layout panel (nullptr -> zeros), advancing by
  // 64 chunks per group.
  __device__ static void run(const uint16_t* const (&a_rows)[kALoads], const uint8_t* const (&b_q)[kBLoads],
                             const uint16_t* const (&b_s)[kBLoads], int K, uint16_t* lds,
                             float16v (&acc)[kTM][kTN]) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    uint16_t* As = lds;
    uint16_t* Bs = lds + BM * kLdsRow;
    const int G = K / kGroup;
    const int KT = (K + kBK - 1) / kBK;

#pragma unroll
    for (int a = 0; a < kTM; ++a)
#pragma unroll
      for (int b = 0; b < kTN; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;

    uint4 areg[kALoads];
    uint4 breg[kBLoads];
    uint16_t sreg[kBLoads];

    auto load = [&](int kt) {
#pragma unroll
      for (int i = 0; i < kALoads; ++i) {
        const int idx = tid + i * kThreads;
        const int col = (idx & 7) * 8;
        const int k = kt * kBK + col;
        areg[i] = (a_rows[i] && k < K) ? *reinterpret_cast<const uint4*>(a_rows[i] + k)
                                       : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < kBLoads; ++i) {
        const int idx = tid + i * kThreads;
        const int cc = (idx >> 6) & 1;
        const int g = kt * 2 + cc;
        if (b_q[i] && g < G) {
          breg[i] = *reinterpret_cast<const uint4*>(b_q[i] + static_cast<int64_t>(g) * 64 * 16);
          sreg[i] = b_s[i][static_cast<int64_t>(g) * 64];
        } else {
          breg[i] = make_uint4(0, 0, 0, 0);
          sreg[i] = 0;
        }
      }
    };

    load(0);
    for (int kt = 0; kt < KT; ++kt) {
      __syncthreads();
#pragma unroll
      for (int i = 0; i < kALoads; ++i) {
        const int idx = tid + i * kThreads;
        const int row = idx >> 3, col = (idx & 7) * 8;
        *reinterpret_cast<uint4*>(As + row * kLdsRow + col) = areg[i];
      }
#pragma unroll
      for (int i = 0; i < kBLoads; ++i) {
        const int idx = tid + i * kThreads;
        const int r = idx & 63, cc = (idx >> 6) & 1, pnl = idx >> 7;
        const int row = pnl * 64 + r;
        uint32_t h[16];
        dequant_chunk_f16(breg[i], sreg[i], h);
        uint4* dst = reinterpret_cast<uint4*>(Bs + row * kLdsRow + cc * 32);
        dst[0] = make_uint4(h[0], h[1], h[2], h[3]);
        dst[1] = make_uint4(h[4], h[5], h[6], h[7]);
        dst[2] = make_uint4(h[8], h[9], h[10], h[11]);
        dst[3] = make_uint4(h[12], h[13], h[14], h[15]);
      }
      __syncthreads();
      if (kt + 1 < KT) load(kt + 1);
#pragma unroll
      for (int ks = 0; ks < kBK / 16; ++ks) {
        half8v af[kTM], bf[kTN];
        const int kofs = ks * 16 + 8 * (lane >> 5);
#pragma unroll
        for (int a = 0; a < kTM; ++a) {
          const int row = wm * (BM / WM) + a * 32 + (lane & 31);
          af[a] = *reinterpret_cast<const half8v*>(As + row * kLdsRow + kofs);
        }
#pragma unroll
        for (int b = 0; b < kTN; ++b) {
          const int row = b_col(wn, b) + (lane & 31);
          bf[b] = *reinterpret_cast<const half8v*>(Bs + row * kLdsRow + kofs);
        }
#pragma unroll
        for (int a = 0; a < kTM; ++a)
#pragma unroll
          for (int b = 0; b < kTN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(af[a], bf[b], acc[a][b], 0, 0, 0);
      }
    }
  }

  // B-row bookkeeping: the thread's i-th B load covers tile row `row` and
  // chunk parity cc; this returns the tile row.
  __device__ static int b_row(int i) {
    const int idx = threadIdx.x + i * kThreads;
    return (idx >> 7) * 64 + (idx & 63);
  }
  __device__ static int b_cc(int i) { return ((threadIdx.x + i * kThreads) >> 6) & 1; }
  __device__ static int a_row(int i) { return (threadIdx.x + i * kThreads) >> 3; }

  // Output coordinates of accumulator register r of tile (a, b) for this lane.
  __device__ static int out_row(int a, int r) {
    const int lane = threadIdx.x & 63;
    const int wm = (threadIdx.x >> 6) / WN;
    return wm * (BM / WM) + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
  __device__ static int out_col(int b) {
    const int lane = threadIdx.x & 63;
    const int wn = (threadIdx.x >> 6) % WN;
    return b_col(wn, b) + (lane & 31);
  }
};

// Pointer to the first chunk (group 0) of row n of a Q4 device-layout matrix
// with G groups; chunk g of that row is at + g * 64 * 16 bytes.
__device__ inline const uint8_t* q4_row_chunk0(const uint8_t* q, int64_t n, int64_t G) {
  return q + ((n / kPanel) * G * kPanel + (n % kPanel)) * 16;
}
__device__ inline const uint16_t* q4_row_scale0(const uint16_t* s, int64_t n, int64_t G) {
  return s + (n / kPanel) * G * kPanel + (n % kPanel);
}

}  // namespace qm
