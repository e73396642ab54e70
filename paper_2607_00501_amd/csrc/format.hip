// Weight format kernels: quantise (fp32 -> canonical codes + fp16 scales),
// dequantise (either layout -> fp32) and repack (canonical <-> device).
//
// These are the offline half of the quantised matmul (BaseRT Sec. 3.3 keeps
// weights in a packed quantised form and dequantises inside the matmul; the
// group-32 symmetric Q4/Q8 formats are the ones evaluated in Sec. 4.1).  One
// thread owns one (matrix, row, group) chunk of 32 weights.  Every kernel is
// bit-exact: the quantiser uses IEEE fp32 division (v_div_scale/fmas/fixup,
// never a reciprocal), v_rndne_f32 (round half to even) and v_cvt_f16_f32
// (round to nearest even, fp16 subnormals kept).
#include "qm_internal.h"

#include <hip/hip_fp16.h>

namespace qm {
namespace {

constexpr int kThreads = 256;

__device__ inline int q4_code_from_canonical(uint32_t byte, int hi) {
  int nib = (byte >> (4 * hi)) & 0xF;
  return nib >= 8 ? nib - 16 : nib;
}

// Offset of the 16-byte device chunk (row n, group g) of one Q4 matrix.
__device__ inline int64_t dev_chunk_q4(int64_t n, int64_t g, int64_t G) {
  return (((n / kPanel) * G + g) * kPanel + (n % kPanel)) * 16;
}
// Offset of the 16-byte half h of the Q8 device chunk (row n, group g).
__device__ inline int64_t dev_half_q8(int64_t n, int64_t g, int64_t G, int h) {
  return (((n / kPanel) * G + g) * 2 + h) * 1024 + (n % kPanel) * 16;
}
__device__ inline int64_t dev_scale(int64_t n, int64_t g, int64_t G) {
  return ((n / kPanel) * G + g) * kPanel + (n % kPanel);
}

// Decode the 32 codes of chunk (n, g) from either layout.
__device__ void load_codes(int32_t fmt, int32_t layout, const uint8_t* q, int64_t n, int64_t g,
                           int64_t G, int64_t K, int codes[32]) {
  if (fmt == QM_Q4_G32) {
    if (layout == QM_LAYOUT_CANONICAL) {
      const uint8_t* p = q + n * (K / 2) + g * 16;
      for (int b = 0; b < 16; ++b) {
        uint32_t v = p[b];
        codes[2 * b] = q4_code_from_canonical(v, 0);
        codes[2 * b + 1] = q4_code_from_canonical(v, 1);
      }
    } else {
      const uint32_t* p = reinterpret_cast<const uint32_t*>(q + dev_chunk_q4(n, g, G));
      for (int j = 0; j < 4; ++j) {
        uint32_t d = p[j];
        for (int t = 0; t < 8; ++t) {
          int off = t < 4 ? 2 * t : 2 * (t - 4) + 1;
          codes[8 * j + off] = static_cast<int>((d >> (4 * t)) & 0xF) - 8;
        }
      }
    }
  } else {
    if (layout == QM_LAYOUT_CANONICAL) {
      const int8_t* p = reinterpret_cast<const int8_t*>(q + n * K + g * 32);
      for (int b = 0; b < 32; ++b) codes[b] = p[b];
    } else {
      for (int h = 0; h < 2; ++h) {
        const uint8_t* p = q + dev_half_q8(n, g, G, h);
        for (int b = 0; b < 16; ++b) codes[16 * h + b] = static_cast<int>(p[b]) - 128;
      }
    }
  }
}

__device__ void store_codes(int32_t fmt, int32_t layout, uint8_t* q, int64_t n, int64_t g, int64_t G,
                            int64_t K, const int codes[32]) {
  if (fmt == QM_Q4_G32) {
    if (layout == QM_LAYOUT_CANONICAL) {
      uint32_t w[4];
      for (int j = 0; j < 4; ++j) {
        uint32_t d = 0;
        for (int b = 0; b < 4; ++b) {
          uint32_t lo = static_cast<uint32_t>(codes[8 * j + 2 * b]) & 0xF;
          uint32_t hi = static_cast<uint32_t>(codes[8 * j + 2 * b + 1]) & 0xF;
          d |= (lo | (hi << 4)) << (8 * b);
        }
        w[j] = d;
      }
      uint4* p = reinterpret_cast<uint4*>(q + n * (K / 2) + g * 16);
      *p = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
      uint32_t w[4];
      for (int j = 0; j < 4; ++j) {
        uint32_t d = 0;
        for (int t = 0; t < 8; ++t) {
          int off = t < 4 ? 2 * t : 2 * (t - 4) + 1;
          d |= (static_cast<uint32_t>(codes[8 * j + off] + 8) & 0xF) << (4 * t);
        }
        w[j] = d;
      }
      uint4* p = reinterpret_cast<uint4*>(q + dev_chunk_q4(n, g, G));
      *p = make_uint4(w[0], w[1], w[2], w[3]);
    }
  } else {
    if (layout == QM_LAYOUT_CANONICAL) {
      uint32_t w[8];
      for (int j = 0; j < 8; ++j) {
        uint32_t d = 0;
        for (int b = 0; b < 4; ++b) d |= (static_cast<uint32_t>(codes[4 * j + b]) & 0xFF) << (8 * b);
        w[j] = d;
      }
      uint4* p = reinterpret_cast<uint4*>(q + n * K + g * 32);
      p[0] = make_uint4(w[0], w[1], w[2], w[3]);
      p[1] = make_uint4(w[4], w[5], w[6], w[7]);
    } else {
      for (int h = 0; h < 2; ++h) {
        uint32_t w[4];
        for (int j = 0; j < 4; ++j) {
          uint32_t d = 0;
          for (int b = 0; b < 4; ++b)
            d |= (static_cast<uint32_t>(codes[16 * h + 4 * j + b] + 128) & 0xFF) << (8 * b);
          w[j] = d;
        }
        *reinterpret_cast<uint4*>(q + dev_half_q8(n, g, G, h)) = make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
  }
}

// ---------------------------------------------------------------- quantise

__global__ __launch_bounds__(kThreads) void quantise_kernel(int32_t fmt, const float* __restrict__ w,
                                                            uint8_t* __restrict__ q,
                                                            uint16_t* __restrict__ s, int64_t rows,
                                                            int64_t K) {
  const int64_t G = K / kGroup;
  const int64_t chunk = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  if (chunk >= rows * G) return;
  const int64_t n = chunk / G;           // row across the whole batch
  const int64_t g = chunk % G;
  const float4* src = reinterpret_cast<const float4*>(w + n * K + g * kGroup);
  float v[32];
  for (int i = 0; i < 8; ++i) {
    float4 t = src[i];
    v[4 * i] = t.x; v[4 * i + 1] = t.y; v[4 * i + 2] = t.z; v[4 * i + 3] = t.w;
  }
  float m = 0.0f;
  for (int i = 0; i < 32; ++i) m = fmaxf(m, fabsf(v[i]));
  const float qmax = fmt == QM_Q4_G32 ? 7.0f : 127.0f;
  const float lo = fmt == QM_Q4_G32 ? -8.0f : -127.0f;
  const float hi = qmax;
  const float s32 = m / qmax;                         // IEEE fp32 division
  const __half s16 = __float2half_rn(s32);
  const float sc = __half2float(s16);
  int codes[32];
  for (int i = 0; i < 32; ++i) {
    float r = sc != 0.0f ? rintf(v[i] / sc) : 0.0f;   // IEEE division, half-even
    r = fminf(fmaxf(r, lo), hi);
    codes[i] = static_cast<int>(r);
  }
  store_codes(fmt, QM_LAYOUT_CANONICAL, q, n, g, G, K, codes);
  s[n * G + g] = __half_as_ushort(s16);
}

// -------------------------------------------------------------- dequantise

__global__ __launch_bounds__(kThreads) void dequantise_kernel(int32_t fmt, int32_t layout,
                                                              const uint8_t* __restrict__ q,
                                                              const uint16_t* __restrict__ s,
                                                              float* __restrict__ out, int64_t batch,
                                                              int64_t N, int64_t K) {
  const int64_t G = K / kGroup;
  const int64_t chunk = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  if (chunk >= batch * N * G) return;
  const int64_t b = chunk / (N * G);
  const int64_t rem = chunk % (N * G);
  const int64_t n = rem / G;
  const int64_t g = rem % G;
  const int64_t rows = matrix_rows(layout, N);
  const uint8_t* qm = q + b * rows * (fmt == QM_Q4_G32 ? K / 2 : K);
  const uint16_t* sm = s + b * rows * G;
  int codes[32];
  load_codes(fmt, layout, qm, n, g, G, K, codes);
  const uint16_t sb = layout == QM_LAYOUT_CANONICAL ? sm[n * G + g] : sm[dev_scale(n, g, G)];
  const float sc = __half2float(__ushort_as_half(sb));
  float4* dst = reinterpret_cast<float4*>(out + (b * N + n) * K + g * kGroup);
  for (int i = 0; i < 8; ++i)
    dst[i] = make_float4(sc * codes[4 * i], sc * codes[4 * i + 1], sc * codes[4 * i + 2],
                         sc * codes[4 * i + 3]);
}

// ------------------------------------------------------------------ repack

// One thread per destination-side chunk.  For CANONICAL -> DEVICE the grid
// covers the padded rows, which are written as zero codes and zero scales.
__global__ __launch_bounds__(kThreads) void repack_kernel(int32_t fmt, int32_t src_layout,
                                                          const uint8_t* __restrict__ sq,
                                                          const uint16_t* __restrict__ ss,
                                                          uint8_t* __restrict__ dq,
                                                          uint16_t* __restrict__ ds, int64_t batch,
                                                          int64_t N, int64_t K) {
  const int64_t G = K / kGroup;
  const int32_t dst_layout = src_layout == QM_LAYOUT_CANONICAL ? QM_LAYOUT_DEVICE : QM_LAYOUT_CANONICAL;
  const int64_t drows = matrix_rows(dst_layout, N);
  const int64_t srows = matrix_rows(src_layout, N);
  const int64_t chunk = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  if (chunk >= batch * drows * G) return;
  const int64_t b = chunk / (drows * G);
  const int64_t rem = chunk % (drows * G);
  const int64_t n = rem / G;
  const int64_t g = rem % G;
  const int64_t rb = fmt == QM_Q4_G32 ? K / 2 : K;
  const uint8_t* sqm = sq + b * srows * rb;
  const uint16_t* ssm = ss + b * srows * G;
  uint8_t* dqm = dq + b * drows * rb;
  uint16_t* dsm = ds + b * drows * G;
  int codes[32];
  uint16_t sb = 0;
  if (n < N) {
    load_codes(fmt, src_layout, sqm, n, g, G, K, codes);
    sb = src_layout == QM_LAYOUT_CANONICAL ? ssm[n * G + g] : ssm[dev_scale(n, g, G)];
  } else {
    // Padding row of the device layout: offset-binary code of 0 is written
    // as raw zero bytes below, so emit the code that encodes to 0x0.
    for (int i = 0; i < 32; ++i) codes[i] = fmt == QM_Q4_G32 ? -8 : -128;
  }
  store_codes(fmt, dst_layout, dqm, n, g, G, K, codes);
  if (dst_layout == QM_LAYOUT_CANONICAL) dsm[n * G + g] = sb;
  else dsm[dev_scale(n, g, G)] = sb;
}

inline unsigned blocks_for(int64_t items) {
  return static_cast<unsigned>((items + kThreads - 1) / kThreads);
}

}  // namespace

hipError_t launch_quantise(int32_t fmt, const float* w, uint8_t* q, uint16_t* s, int64_t batch,
                           int64_t n, int64_t k, hipStream_t st) {
  const int64_t items = batch * n * (k / kGroup);
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(quantise_kernel, dim3(blocks_for(items)), dim3(kThreads), 0, st, fmt, w, q, s,
                     batch * n, k);
  return hipGetLastError();
}

hipError_t launch_dequantise(int32_t fmt, int32_t layout, const uint8_t* q, const uint16_t* s,
                             float* out, int64_t batch, int64_t n, int64_t k, hipStream_t st) {
  const int64_t items = batch * n * (k / kGroup);
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(dequantise_kernel, dim3(blocks_for(items)), dim3(kThreads), 0, st, fmt, layout,
                     q, s, out, batch, n, k);
  return hipGetLastError();
}

hipError_t launch_repack(int32_t fmt, int32_t src_layout, const uint8_t* sq, const uint16_t* ss,
                         uint8_t* dq, uint16_t* ds, int64_t batch, int64_t n, int64_t k,
                         hipStream_t st) {
  const int32_t dst_layout = src_layout == QM_LAYOUT_CANONICAL ? QM_LAYOUT_DEVICE : QM_LAYOUT_CANONICAL;
  const int64_t items = batch * matrix_rows(dst_layout, n) * (k / kGroup);
  if (items == 0) return hipSuccess;
  hipLaunchKernelGGL(repack_kernel, dim3(blocks_for(items)), dim3(kThreads), 0, st, fmt, src_layout,
                     sq, ss, dq, ds, batch, n, k);
  return hipGetLastError();
}

}  // namespace qm
