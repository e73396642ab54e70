// Weight format kernels: quantise (fp32 -> canonical codes + fp16 scales),
// dequantise (either layout -> fp32) and repack (canonical <-> device).
//
// These are the offline half of the quantised matmul (BaseRT Sec. 3.3 keeps
// weights in a packed quantised form and dequantises inside the matmul;
// Sec. 4.1 lists the eight formats, Q2 .. Q8, BF16 and FP16).  One
// thread owns one (matrix, row, group) chunk of 32 weights.  Every kernel is
// bit-exact: the quantiser uses IEEE fp32 division (v_div_scale/fmas/fixup,
// never a reciprocal), v_rndne_f32 (round half to even) and v_cvt_f16_f32
// (round to nearest even, fp16 subnormals kept).
#include "qm_internal.h"

#include <hip/hip_fp16.h>

namespace qm {
namespace {

constexpr int kThreads = 256;

// Device layout addressing (one (panel, group) chunk block per CB bytes).
__device__ inline const uint8_t* dev_block(const uint8_t* q, int32_t fmt, int64_t n, int64_t g, int64_t G) {
  return q + ((n / kPanel) * G + g) * chunk_block_bytes(fmt);
}
__device__ inline int64_t dev_scale(int64_t n, int64_t g, int64_t G) {
  return ((n / kPanel) * G + g) * kPanel + (n % kPanel);
}

// Positions of code k (0..31 of a group) inside the planes of a row:
// nibble plane dword k/8, nibble slot 2t -> t, 2t+1 -> 4+t of the dword's k
// offset; crumb plane dword k/16, bits 2(k%16/2) (+16 for odd k); bit plane
// bit k/2 (+16 for odd k).
__device__ inline int nib_shift(int k) { const int o = k % 8; return 4 * (o % 2 == 0 ? o / 2 : 4 + o / 2); }
__device__ inline int crumb_shift(int k) { const int o = k % 16; return 2 * (o / 2) + (o % 2 ? 16 : 0); }
__device__ inline int bit_shift(int k) { return k / 2 + (k % 2 ? 16 : 0); }

// Plane composition of the bit-plane formats: (low plane, high plane, bits of the low part).
struct Planes { int low; int high; int low_bits; };   // 0 none, 1 nibble, 2 crumb, 3 bit
__device__ inline Planes planes_of(int32_t fmt) {
  switch (fmt) {
    case QM_Q2_G32: return {2, 0, 2};
    case QM_Q3_G32: return {2, 3, 2};
    case QM_Q5_G32: return {1, 3, 4};
    default: return {1, 2, 4};                         // Q6
  }
}
__device__ inline int plane_row_bytes(int plane) { return plane == 1 ? 16 : plane == 2 ? 8 : 4; }
__device__ inline int plane_shift(int plane, int k) {
  return plane == 1 ? nib_shift(k) : plane == 2 ? crumb_shift(k) : bit_shift(k);
}
__device__ inline int plane_dword(int plane, int k) { return plane == 1 ? k / 8 : plane == 2 ? k / 16 : 0; }
__device__ inline uint32_t plane_mask(int plane) { return plane == 1 ? 0xFu : plane == 2 ? 0x3u : 0x1u; }

// Decode the 32 codes of chunk (n, g) from either layout: signed codes for
// the integer formats, the uint16 patterns for F16/BF16.
__device__ void load_codes(int32_t fmt, int32_t layout, const uint8_t* q, int64_t n, int64_t g,
                           int64_t G, int64_t K, int codes[32]) {
  const int b = fmt_bits(fmt);
  if (fmt_float(fmt)) {
    if (layout == QM_LAYOUT_CANONICAL) {
      const uint16_t* p = reinterpret_cast<const uint16_t*>(q) + n * K + g * kGroup;
      for (int k = 0; k < 32; ++k) codes[k] = p[k];
    } else {
      const uint8_t* blk = dev_block(q, fmt, n, g, G);
      for (int k = 0; k < 32; ++k)
        codes[k] = reinterpret_cast<const uint16_t*>(blk + (k / 8) * 1024 + (n % kPanel) * 16)[k % 8];
    }
    return;
  }
  if (layout == QM_LAYOUT_CANONICAL) {
    // Little-endian bit stream of the row; the group starts at byte 4b*g.
    const uint32_t* p = reinterpret_cast<const uint32_t*>(q + n * row_code_bytes(fmt, K) + g * 4 * b);
    for (int k = 0; k < 32; ++k) {
      uint32_t field = 0;
      for (int i = 0; i < b; ++i) {
        const int pos = b * k + i;
        field |= ((p[pos / 32] >> (pos % 32)) & 1u) << i;
      }
      codes[k] = field >= (1u << (b - 1)) ? static_cast<int>(field) - (1 << b) : static_cast<int>(field);
    }
    return;
  }
  const uint8_t* blk = dev_block(q, fmt, n, g, G);
  const int r = static_cast<int>(n % kPanel);
  const int bias = 1 << (b - 1);
  if (fmt == QM_Q8_G32) {
    for (int k = 0; k < 32; ++k) codes[k] = static_cast<int>(blk[(k / 16) * 1024 + r * 16 + k % 16]) - 128;
    return;
  }
  if (fmt == QM_Q4_G32) {
    const uint32_t* p = reinterpret_cast<const uint32_t*>(blk + r * 16);
    for (int k = 0; k < 32; ++k) codes[k] = static_cast<int>((p[k / 8] >> nib_shift(k)) & 0xF) - bias;
    return;
  }
  const Planes pl = planes_of(fmt);
  const int lo_bytes = 64 * plane_row_bytes(pl.low);
  const uint32_t* lo = reinterpret_cast<const uint32_t*>(blk + r * plane_row_bytes(pl.low));
  const uint32_t* hi = pl.high ? reinterpret_cast<const uint32_t*>(blk + lo_bytes + r * plane_row_bytes(pl.high))
                               : nullptr;
  for (int k = 0; k < 32; ++k) {
    uint32_t u = (lo[plane_dword(pl.low, k)] >> plane_shift(pl.low, k)) & plane_mask(pl.low);
    if (hi) u |= ((hi[plane_dword(pl.high, k)] >> plane_shift(pl.high, k)) & plane_mask(pl.high)) << pl.low_bits;
    codes[k] = static_cast<int>(u) - bias;
  }
}

__device__ void store_codes(int32_t fmt, int32_t layout, uint8_t* q, int64_t n, int64_t g, int64_t G,
                            int64_t K, const int codes[32]) {
  const int b = fmt_bits(fmt);
  if (fmt_float(fmt)) {
    if (layout == QM_LAYOUT_CANONICAL) {
      uint16_t* p = reinterpret_cast<uint16_t*>(q) + n * K + g * kGroup;
      for (int k = 0; k < 32; ++k) p[k] = static_cast<uint16_t>(codes[k]);
    } else {
      uint8_t* blk = q + ((n / kPanel) * G + g) * chunk_block_bytes(fmt);
      for (int j = 0; j < 4; ++j) {
        uint32_t w[4];
        for (int i = 0; i < 4; ++i)
          w[i] = static_cast<uint32_t>(codes[8 * j + 2 * i] & 0xFFFF) |
                 (static_cast<uint32_t>(codes[8 * j + 2 * i + 1] & 0xFFFF) << 16);
        *reinterpret_cast<uint4*>(blk + j * 1024 + (n % kPanel) * 16) = make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
    return;
  }
  if (layout == QM_LAYOUT_CANONICAL) {
    uint32_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int k = 0; k < 32; ++k) {
      const uint32_t field = static_cast<uint32_t>(codes[k]) & ((1u << b) - 1);
      for (int i = 0; i < b; ++i) {
        const int pos = b * k + i;
        w[pos / 32] |= ((field >> i) & 1u) << (pos % 32);
      }
    }
    uint32_t* p = reinterpret_cast<uint32_t*>(q + n * row_code_bytes(fmt, K) + g * 4 * b);
    for (int i = 0; i < b; ++i) p[i] = w[i];
    return;
  }
  uint8_t* blk = q + ((n / kPanel) * G + g) * chunk_block_bytes(fmt);
  const int r = static_cast<int>(n % kPanel);
  const int bias = 1 << (b - 1);
  if (fmt == QM_Q8_G32) {
    for (int h = 0; h < 2; ++h) {
      uint32_t w[4];
      for (int j = 0; j < 4; ++j) {
        uint32_t d = 0;
        for (int i = 0; i < 4; ++i) d |= (static_cast<uint32_t>(codes[16 * h + 4 * j + i] + 128) & 0xFF) << (8 * i);
        w[j] = d;
      }
      *reinterpret_cast<uint4*>(blk + h * 1024 + r * 16) = make_uint4(w[0], w[1], w[2], w[3]);
    }
    return;
  }
  if (fmt == QM_Q4_G32) {
    uint32_t w[4] = {0, 0, 0, 0};
    for (int k = 0; k < 32; ++k) w[k / 8] |= (static_cast<uint32_t>(codes[k] + bias) & 0xF) << nib_shift(k);
    *reinterpret_cast<uint4*>(blk + r * 16) = make_uint4(w[0], w[1], w[2], w[3]);
    return;
  }
  const Planes pl = planes_of(fmt);
  uint32_t lo[4] = {0, 0, 0, 0}, hi[4] = {0, 0, 0, 0};
  for (int k = 0; k < 32; ++k) {
    const uint32_t u = static_cast<uint32_t>(codes[k] + bias) & ((1u << b) - 1);
    lo[plane_dword(pl.low, k)] |= (u & plane_mask(pl.low)) << plane_shift(pl.low, k);
    if (pl.high) hi[plane_dword(pl.high, k)] |= ((u >> pl.low_bits) & plane_mask(pl.high)) << plane_shift(pl.high, k);
  }
  const int lo_row = plane_row_bytes(pl.low);
  uint32_t* plo = reinterpret_cast<uint32_t*>(blk + r * lo_row);
  for (int i = 0; i < lo_row / 4; ++i) plo[i] = lo[i];
  if (pl.high) {
    const int hi_row = plane_row_bytes(pl.high);
    uint32_t* phi = reinterpret_cast<uint32_t*>(blk + 64 * lo_row + r * hi_row);
    for (int i = 0; i < hi_row / 4; ++i) phi[i] = hi[i];
  }
}

// fp32 -> bf16 pattern, round to nearest even (finite inputs).
__device__ inline uint16_t bf16_rne(float v) {
  const uint32_t u = __float_as_uint(v);
  const uint32_t keep = u >> 16, rest = u & 0xFFFFu;
  const uint32_t up = (rest > 0x8000u || (rest == 0x8000u && (keep & 1u))) ? 1u : 0u;
  return static_cast<uint16_t>(keep + up);
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
  int codes[32];
  if (fmt_float(fmt)) {
    for (int i = 0; i < 32; ++i)
      codes[i] = fmt == QM_F16 ? __half_as_ushort(__float2half_rn(v[i])) : bf16_rne(v[i]);
    store_codes(fmt, QM_LAYOUT_CANONICAL, q, n, g, G, K, codes);
    return;
  }
  float m = 0.0f;
  for (int i = 0; i < 32; ++i) m = fmaxf(m, fabsf(v[i]));
  const int b = fmt_bits(fmt);
  const float qmax = fmt == QM_Q8_G32 ? 127.0f : static_cast<float>((1 << (b - 1)) - 1);
  const float lo = fmt == QM_Q8_G32 ? -127.0f : -static_cast<float>(1 << (b - 1));
  const float hi = qmax;
  const float s32 = m / qmax;                         // IEEE fp32 division
  const __half s16 = __float2half_rn(s32);
  const float sc = __half2float(s16);
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
  const uint8_t* qm = q + b * rows * row_code_bytes(fmt, K);
  int codes[32];
  load_codes(fmt, layout, qm, n, g, G, K, codes);
  float val[32];
  if (fmt_float(fmt)) {
    for (int i = 0; i < 32; ++i)
      val[i] = fmt == QM_F16 ? __half2float(__ushort_as_half(static_cast<uint16_t>(codes[i])))
                             : __uint_as_float(static_cast<uint32_t>(codes[i]) << 16);
  } else {
    const uint16_t* sm = s + b * rows * G;
    const uint16_t sb = layout == QM_LAYOUT_CANONICAL ? sm[n * G + g] : sm[dev_scale(n, g, G)];
    const float sc = __half2float(__ushort_as_half(sb));
    for (int i = 0; i < 32; ++i) val[i] = sc * codes[i];
  }
  float4* dst = reinterpret_cast<float4*>(out + (b * N + n) * K + g * kGroup);
  for (int i = 0; i < 8; ++i) dst[i] = make_float4(val[4 * i], val[4 * i + 1], val[4 * i + 2], val[4 * i + 3]);
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
  const int64_t rb = row_code_bytes(fmt, K);
  const bool scaled = !fmt_float(fmt);
  const uint8_t* sqm = sq + b * srows * rb;
  uint8_t* dqm = dq + b * drows * rb;
  int codes[32];
  uint16_t sb = 0;
  if (n < N) {
    load_codes(fmt, src_layout, sqm, n, g, G, K, codes);
    if (scaled) {
      const uint16_t* ssm = ss + b * srows * G;
      sb = src_layout == QM_LAYOUT_CANONICAL ? ssm[n * G + g] : ssm[dev_scale(n, g, G)];
    }
  } else {
    // Padding row of the device layout: zero bytes.  For the integer
    // formats that is the offset-binary code of -2^(b-1) (Q8: -128).
    for (int i = 0; i < 32; ++i) codes[i] = scaled ? -(1 << (fmt_bits(fmt) - 1)) : 0;
  }
  store_codes(fmt, dst_layout, dqm, n, g, G, K, codes);
  if (scaled) {
    uint16_t* dsm = ds + b * drows * G;
    if (dst_layout == QM_LAYOUT_CANONICAL) dsm[n * G + g] = sb;
    else dsm[dev_scale(n, g, G)] = sb;
  }
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
