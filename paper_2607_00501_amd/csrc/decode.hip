// The small kernels that join the matmuls and attention of one decode step
// into a whole token (BaseRT Sec. 3.2: normalisation, RoPE, embedding and
// sampling kernels beside the matmul and attention ones): embedding gather,
// RMSNorm with the residual add folded in, rotary embedding fused with the
// KV-cache append, fp32 -> fp16 conversion of a matmul input, and greedy
// sampling.  Each moves a few KiB per token; they are latency-bound, so each
// is one launch sized to the data, with no host synchronisation anywhere, so
// the token id stays on the device from the argmax to the next embedding.
#include <cmath>

#include "qm_internal.h"
#include "rope.h"

namespace qm {
namespace {

__device__ __forceinline__ float h2f(uint16_t b) {
  _Float16 h;
  __builtin_memcpy(&h, &b, 2);
  return static_cast<float>(h);
}
__device__ __forceinline__ uint16_t f2h(float f) {
  const _Float16 h = static_cast<_Float16>(f);   // round to nearest even
  uint16_t b;
  __builtin_memcpy(&b, &h, 2);
  return b;
}

// Sum over the 256 threads of a workgroup (4 wavefronts).
__device__ __forceinline__ float block_sum(float v, float* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  v = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return v;
}

__global__ __launch_bounds__(256) void embed_kernel(const uint16_t* __restrict__ table, int64_t vocab,
                                                    int64_t hidden, const int32_t* __restrict__ token,
                                                    float* __restrict__ x) {
  const int32_t t = *token;
  const bool ok = t >= 0 && t < vocab;
  const uint16_t* row = table + (ok ? t : 0) * hidden;
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < hidden; i += gridDim.x * 256)
    x[i] = ok ? h2f(row[i]) : __builtin_nanf("");
}

// One workgroup per row: x += residual (written back), out = fp16(x / rms * w).
// Rows of up to 256 * PER elements stay in registers: the loads of x, the
// residual and w go out together, so a row costs one memory round trip
// before the reduction.
template <int PER>
__global__ __launch_bounds__(256) void rmsnorm_reg_kernel(float* __restrict__ x, const float* __restrict__ res,
                                                          const uint16_t* __restrict__ w, int64_t hidden, float eps,
                                                          uint16_t* __restrict__ out) {
  __shared__ float red[4];
  float* xr = x + blockIdx.x * hidden;
  const float* rr = res ? res + blockIdx.x * hidden : nullptr;
  float v[PER], g[PER], r[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int i = threadIdx.x + j * 256;
    v[j] = i < hidden ? xr[i] : 0.0f;
    g[j] = i < hidden ? h2f(w[i]) : 0.0f;
    r[j] = rr && i < hidden ? rr[i] : 0.0f;
  }
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    v[j] += r[j];
    ss = fmaf(v[j], v[j], ss);
  }
  if (rr) {
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (threadIdx.x + j * 256 < hidden) xr[threadIdx.x + j * 256] = v[j];
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(hidden) + eps);
  uint16_t* o = out + blockIdx.x * hidden;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (threadIdx.x + j * 256 < hidden) o[threadIdx.x + j * 256] = f2h(v[j] * inv * g[j]);
}

// The same with 16-byte loads (four elements of x and of the residual, four
// gains, per load) when hidden % 4 == 0 and the rows are 16-byte aligned:
// a quarter of the load instructions, which is what bounds a lone
// workgroup's row.
template <int P4>
__global__ __launch_bounds__(256) void rmsnorm_vec_kernel(float* __restrict__ x, const float* __restrict__ res,
                                                          const uint16_t* __restrict__ w, int64_t hidden, float eps,
                                                          uint16_t* __restrict__ out) {
  __shared__ float red[4];
  const int n4 = static_cast<int>(hidden / 4);
  float4* xr = reinterpret_cast<float4*>(x + blockIdx.x * hidden);
  const float4* rr = res ? reinterpret_cast<const float4*>(res + blockIdx.x * hidden) : nullptr;
  const uint2* wr = reinterpret_cast<const uint2*>(w);
  float4 v[P4], r[P4];
  uint2 g[P4];
#pragma unroll
  for (int j = 0; j < P4; ++j) {
    const int i = threadIdx.x + j * 256;
    const bool ok = i < n4;
    v[j] = ok ? xr[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    g[j] = ok ? wr[i] : make_uint2(0u, 0u);
    r[j] = rr && ok ? rr[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < P4; ++j) {
    v[j].x += r[j].x; v[j].y += r[j].y; v[j].z += r[j].z; v[j].w += r[j].w;
    ss = fmaf(v[j].x, v[j].x, ss);
    ss = fmaf(v[j].y, v[j].y, ss);
    ss = fmaf(v[j].z, v[j].z, ss);
    ss = fmaf(v[j].w, v[j].w, ss);
  }
  if (rr) {
#pragma unroll
    for (int j = 0; j < P4; ++j)
      if (threadIdx.x + j * 256 < n4) xr[threadIdx.x + j * 256] = v[j];
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(hidden) + eps);
  uint2* o = reinterpret_cast<uint2*>(out + blockIdx.x * hidden);
#pragma unroll
  for (int j = 0; j < P4; ++j) {
    const int i = threadIdx.x + j * 256;
    if (i < n4) {
      const uint32_t a = f2h(v[j].x * inv * h2f(static_cast<uint16_t>(g[j].x))) |
                         static_cast<uint32_t>(f2h(v[j].y * inv * h2f(static_cast<uint16_t>(g[j].x >> 16)))) << 16;
      const uint32_t b = f2h(v[j].z * inv * h2f(static_cast<uint16_t>(g[j].y))) |
                         static_cast<uint32_t>(f2h(v[j].w * inv * h2f(static_cast<uint16_t>(g[j].y >> 16)))) << 16;
      o[i] = make_uint2(a, b);
    }
  }
}

// Rows longer than the register tile: two passes over the row.
__global__ __launch_bounds__(256) void rmsnorm_kernel(float* __restrict__ x, const float* __restrict__ res,
                                                      const uint16_t* __restrict__ w, int64_t hidden, float eps,
                                                      uint16_t* __restrict__ out) {
  __shared__ float red[4];
  float* xr = x + blockIdx.x * hidden;
  const float* rr = res ? res + blockIdx.x * hidden : nullptr;
  float ss = 0.0f;
  for (int64_t i = threadIdx.x; i < hidden; i += 256) {
    float v = xr[i];
    if (rr) {
      v += rr[i];
      xr[i] = v;
    }
    ss = fmaf(v, v, ss);
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(hidden) + eps);
  uint16_t* o = out + blockIdx.x * hidden;
  for (int64_t i = threadIdx.x; i < hidden; i += 256) o[i] = f2h(xr[i] * inv * h2f(w[i]));
}

// Per-head RMSNorm before RoPE (the Qwen3 layer): thread i of the head's
// D/2 threads holds dimensions i and i + D/2.
__device__ __forceinline__ void head_rmsnorm(float& a, float& b, int i, int half, const uint16_t* __restrict__ gain,
                                             float eps) {
  float ss = fmaf(a, a, b * b);
  for (int off = half / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off, half);
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(2 * half) + eps);
  a = a * inv * h2f(gain[i]);
  b = b * inv * h2f(gain[i + half]);
}

// One workgroup of D/2 threads per head: heads [0, hq) are queries (rotated
// into q_out), [hq, hq + hkv) keys (rotated into the key cache at row pos),
// the rest values (copied into the value cache at row pos).  Thread i
// rotates the pair (i, i + D/2) by pos * theta^(-2i/D); the angle and its
// sine and cosine are taken in fp64 so that they stay exact to fp32 at
// positions in the hundreds of thousands.
__global__ void rope_append_kernel(const float* __restrict__ q, const float* __restrict__ k,
                                   const float* __restrict__ v, int hq, int hkv, int d, int64_t pos,
                                   int64_t max_len, double log2_theta, uint16_t* __restrict__ q_out,
                                   uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                   const uint16_t* __restrict__ q_gain, const uint16_t* __restrict__ k_gain,
                                   float eps, const float2* __restrict__ table) {
  const int h = blockIdx.x, i = threadIdx.x, half = d / 2;
  if (h >= hq + hkv) {
    const int kh = h - hq - hkv;
    uint16_t* dst = vc + (static_cast<int64_t>(kh) * max_len + pos) * d;
    dst[i] = f2h(v[kh * d + i]);
    dst[i + half] = f2h(v[kh * d + i + half]);
    return;
  }
  const float2 cs = table ? table[pos * half + i] : rope_cos_sin(pos, i, d, log2_theta);   // same values
  const float c = cs.x, s = cs.y;
  const float* src = h < hq ? q + h * d : k + (h - hq) * d;
  uint16_t* dst = h < hq ? q_out + h * d : kc + (static_cast<int64_t>(h - hq) * max_len + pos) * d;
  float a = src[i], b = src[i + half];
  if (q_gain) head_rmsnorm(a, b, i, half, h < hq ? q_gain : k_gain, eps);
  dst[i] = f2h(rope_low(a, b, c, s));
  dst[i + half] = f2h(rope_high(a, b, c, s));
}

// table[p][i] = (cos, sin) of the angle of pair i at position p, for every
// position of a cache (built once; the same function as the kernels above).
__global__ __launch_bounds__(256) void rope_table_kernel(int64_t max_len, int d, double log2_theta,
                                                         float2* __restrict__ table) {
  const int64_t n = max_len * (d / 2);
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < n; e += static_cast<int64_t>(gridDim.x) * 256)
    table[e] = rope_cos_sin(e / (d / 2), static_cast<int>(e % (d / 2)), d, log2_theta);
}

// The same table with the frequencies of the Llama 3 long-context rule.
__global__ __launch_bounds__(256) void rope_table_llama3_kernel(int64_t max_len, int d, double log2_theta,
                                                                double factor, double low, double high, double orig,
                                                                float2* __restrict__ table) {
#pragma clang fp contract(off)
  const int64_t n = max_len * (d / 2);
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < n; e += static_cast<int64_t>(gridDim.x) * 256) {
    const double ang = static_cast<double>(e / (d / 2)) *
                       rope_freq_llama3(static_cast<int>(e % (d / 2)), d, log2_theta, factor, low, high, orig);
    table[e] = make_float2(static_cast<float>(cos(ang)), static_cast<float>(sin(ang)));
  }
}

// Prompt (prefill) glue: the same operations over m tokens.
// x[r] = table[tokens[r]] (NaN rows for ids outside the vocabulary).
__global__ __launch_bounds__(256) void embed_rows_kernel(const uint16_t* __restrict__ table, int64_t vocab,
                                                         int64_t hidden, const int32_t* __restrict__ tokens,
                                                         float* __restrict__ x) {
  const int64_t r = blockIdx.x;
  const int32_t t = tokens[r];
  const bool ok = t >= 0 && t < vocab;
  const uint16_t* row = table + (ok ? t : 0) * hidden;
  for (int64_t i = threadIdx.x; i < hidden; i += 256) x[r * hidden + i] = ok ? h2f(row[i]) : __builtin_nanf("");
}

// Grid (head, token): token r at position p0 + r.  Inputs are the projection
// outputs [m][heads * D] (each head's dimensions interleaved when
// `interleaved`: column 2i = dimension i, 2i + 1 = dimension i + D/2);
// queries go to q_out [Hq][m][D] (the prefill attention's layout), keys and
// values to cache rows p0 + r.
__global__ void rope_append_rows_kernel(const float* __restrict__ q, const float* __restrict__ k,
                                        const float* __restrict__ v, int hq, int hkv, int d, int64_t m, int64_t p0,
                                        int64_t max_len, double log2_theta, int interleaved,
                                        uint16_t* __restrict__ q_out, uint16_t* __restrict__ kc,
                                        uint16_t* __restrict__ vc, const uint16_t* __restrict__ q_gain,
                                        const uint16_t* __restrict__ k_gain, float eps,
                                        const float2* __restrict__ table) {
  const int h = blockIdx.x, i = threadIdx.x, half = d / 2;
  const int64_t r = blockIdx.y, pos = p0 + r;
  if (h >= hq + hkv) {
    const int kh = h - hq - hkv;
    const float* src = v + r * hkv * d + kh * d;
    uint16_t* dst = vc + (static_cast<int64_t>(kh) * max_len + pos) * d;
    dst[i] = f2h(src[i]);
    dst[i + half] = f2h(src[i + half]);
    return;
  }
  // (cos, sin) from the cache's table when given (the same values, built
  // once by rope_table_kernel), else computed here.
  const float2 cs = table ? table[pos * half + i] : rope_cos_sin(pos, i, d, log2_theta);
  const float* src = h < hq ? q + r * hq * d + h * d : k + r * hkv * d + (h - hq) * d;
  uint16_t* dst = h < hq ? q_out + (static_cast<int64_t>(h) * m + r) * d
                         : kc + (static_cast<int64_t>(h - hq) * max_len + pos) * d;
  float a = interleaved ? src[2 * i] : src[i], b = interleaved ? src[2 * i + 1] : src[i + half];
  if (q_gain) head_rmsnorm(a, b, i, half, h < hq ? q_gain : k_gain, eps);
  dst[i] = f2h(rope_low(a, b, cs.x, cs.y));
  dst[i + half] = f2h(rope_high(a, b, cs.x, cs.y));
}

// o [H][m][D] fp32 -> out [m][H * D] fp16 (the output projection's input).
__global__ __launch_bounds__(256) void heads_to_rows_kernel(const float* __restrict__ o, int h, int64_t m, int d,
                                                            uint16_t* __restrict__ out) {
  const int64_t n = static_cast<int64_t>(h) * m * d;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < n; e += static_cast<int64_t>(gridDim.x) * 256) {
    const int64_t r = e / (static_cast<int64_t>(h) * d), c = e % (static_cast<int64_t>(h) * d);
    out[e] = f2h(o[((c / d) * m + r) * d + c % d]);
  }
}

// out = fp16(silu(g) * u) elementwise.
__global__ __launch_bounds__(256) void swiglu_kernel(const float* __restrict__ g, const float* __restrict__ u,
                                                     int64_t n, uint16_t* __restrict__ out) {
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < n; e += static_cast<int64_t>(gridDim.x) * 256) {
    const float a = g[e];
    out[e] = f2h(a / (1.0f + expf(-a)) * u[e]);
  }
}

__global__ __launch_bounds__(256) void cast_f16_kernel(const float* __restrict__ x, int64_t n,
                                                       uint16_t* __restrict__ y) {
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) y[i] = f2h(x[i]);
}

// Greedy sampling: index of the largest logit, the lowest index among equal
// ones; NaNs are never chosen; 0 if every logit is NaN.  Pass 1: each of up
// to kArgmaxBlocks workgroups reduces a strided share of the logits, four
// independent loads in flight per lane, to one (value, index) pair (a lone
// workgroup writes the token directly); pass 2 reduces the pairs.
constexpr int kArgmaxBlocks = 256;

// (value, index) pair order: larger value first, then lower index; the
// index INT32_MAX marks "nothing seen yet".
__device__ __forceinline__ void take_better(float& bv, int32_t& bi, float v, int32_t i) {
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

__device__ __forceinline__ void block_best(float& bv, int32_t& bi) {
  __shared__ float sv[4];
  __shared__ int32_t si[4];
  for (int o = 32; o > 0; o >>= 1) take_better(bv, bi, __shfl_xor(bv, o, 64), __shfl_xor(bi, o, 64));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sv[w] = bv;
    si[w] = bi;
  }
  __syncthreads();
  bv = sv[0];
  bi = si[0];
  for (int j = 1; j < 4; ++j) take_better(bv, bi, sv[j], si[j]);
}

__global__ __launch_bounds__(256) void argmax_partial_kernel(const float* __restrict__ x, int64_t n,
                                                             float* __restrict__ pv, int32_t* __restrict__ pi,
                                                             int32_t* __restrict__ token) {
  float best = -INFINITY;
  int32_t idx = INT32_MAX;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int64_t base = blockIdx.x * 256 + threadIdx.x; base < n; base += 4 * stride) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t i = base + u * stride;
      v[u] = i < n ? x[i] : __builtin_nanf("");
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {   // increasing indices: keep the first of equal values
      if (v[u] > best || (v[u] == best && idx == INT32_MAX)) {
        best = v[u];
        idx = static_cast<int32_t>(base + u * stride);
      }
    }
  }
  block_best(best, idx);
  if (threadIdx.x == 0) {
    if (gridDim.x == 1) {
      token[0] = idx == INT32_MAX ? 0 : idx;
    } else {
      pv[blockIdx.x] = best;
      pi[blockIdx.x] = idx;
    }
  }
}

__global__ __launch_bounds__(256) void argmax_final_kernel(const float* __restrict__ pv,
                                                           const int32_t* __restrict__ pi, int nb,
                                                           int32_t* __restrict__ token) {
  float best = -INFINITY;
  int32_t idx = INT32_MAX;
  if (static_cast<int>(threadIdx.x) < nb) {
    best = pv[threadIdx.x];
    idx = pi[threadIdx.x];
  }
  block_best(best, idx);
  if (threadIdx.x == 0) token[0] = idx == INT32_MAX ? 0 : idx;
}

unsigned spread_blocks(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return static_cast<unsigned>(b < 1024 ? (b < 1 ? 1 : b) : 1024);
}

}  // namespace

hipError_t launch_embed(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* token, float* x,
                        hipStream_t st) {
  hipLaunchKernelGGL(embed_kernel, dim3(spread_blocks(hidden)), dim3(256), 0, st, table, vocab, hidden, token, x);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(float* x, const float* res, const uint16_t* w, int64_t rows, int64_t hidden, float eps,
                          uint16_t* out, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(rows)), block(256);
  const bool vec = hidden % 4 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(res) & 15) == 0 && (reinterpret_cast<uintptr_t>(w) & 7) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 7) == 0;
  if (vec && hidden <= 1024 * 2) {
    hipLaunchKernelGGL(rmsnorm_vec_kernel<2>, grid, block, 0, st, x, res, w, hidden, eps, out);
    return hipGetLastError();
  }
  if (vec && hidden <= 1024 * 4) {
    hipLaunchKernelGGL(rmsnorm_vec_kernel<4>, grid, block, 0, st, x, res, w, hidden, eps, out);
    return hipGetLastError();
  }
  if (vec && hidden <= 1024 * 8) {
    hipLaunchKernelGGL(rmsnorm_vec_kernel<8>, grid, block, 0, st, x, res, w, hidden, eps, out);
    return hipGetLastError();
  }
  if (hidden <= 256 * 4) {
    hipLaunchKernelGGL(rmsnorm_reg_kernel<4>, grid, block, 0, st, x, res, w, hidden, eps, out);
    return hipGetLastError();
  }
  if (hidden <= 256 * 8) {
    hipLaunchKernelGGL(rmsnorm_reg_kernel<8>, grid, block, 0, st, x, res, w, hidden, eps, out);
    return hipGetLastError();
  }
  if (hidden <= 256 * 16) {
    hipLaunchKernelGGL(rmsnorm_reg_kernel<16>, grid, block, 0, st, x, res, w, hidden, eps, out);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(static_cast<unsigned>(rows)), dim3(256), 0, st, x, res, w, hidden, eps,
                     out);
  return hipGetLastError();
}

hipError_t launch_rope_append(const float* q, const float* k, const float* v, int32_t hq, int32_t hkv, int32_t d,
                              int64_t pos, int64_t max_len, float theta, uint16_t* q_out, uint16_t* kc,
                              uint16_t* vc, const uint16_t* q_gain, const uint16_t* k_gain, float eps,
                              const float* table, hipStream_t st) {
  hipLaunchKernelGGL(rope_append_kernel, dim3(static_cast<unsigned>(hq + 2 * hkv)), dim3(d / 2), 0, st, q, k, v,
                     hq, hkv, d, pos, max_len, std::log2(static_cast<double>(theta)), q_out, kc, vc, q_gain, k_gain,
                     eps, reinterpret_cast<const float2*>(table));
  return hipGetLastError();
}

hipError_t launch_rope_table(int64_t max_len, int32_t d, float theta, float* table, hipStream_t st) {
  hipLaunchKernelGGL(rope_table_kernel, dim3(spread_blocks(max_len * (d / 2))), dim3(256), 0, st, max_len, d,
                     std::log2(static_cast<double>(theta)), reinterpret_cast<float2*>(table));
  return hipGetLastError();
}

hipError_t launch_rope_table_llama3(int64_t max_len, int32_t d, float theta, float factor, float low, float high,
                                    float orig, float* table, hipStream_t st) {
  hipLaunchKernelGGL(rope_table_llama3_kernel, dim3(spread_blocks(max_len * (d / 2))), dim3(256), 0, st, max_len, d,
                     std::log2(static_cast<double>(theta)), static_cast<double>(factor), static_cast<double>(low),
                     static_cast<double>(high), static_cast<double>(orig), reinterpret_cast<float2*>(table));
  return hipGetLastError();
}

hipError_t launch_embed_rows(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* tokens, int64_t m,
                             float* x, hipStream_t st) {
  if (m == 0) return hipSuccess;
  hipLaunchKernelGGL(embed_rows_kernel, dim3(static_cast<unsigned>(m)), dim3(256), 0, st, table, vocab, hidden, tokens,
                     x);
  return hipGetLastError();
}

hipError_t launch_rope_append_rows(const float* q, const float* k, const float* v, int32_t hq, int32_t hkv, int32_t d,
                                   int64_t m, int64_t p0, int64_t max_len, float theta, int32_t interleaved,
                                   uint16_t* q_out, uint16_t* kc, uint16_t* vc, const uint16_t* q_gain,
                                   const uint16_t* k_gain, float eps, const float* table, hipStream_t st) {
  hipLaunchKernelGGL(rope_append_rows_kernel, dim3(static_cast<unsigned>(hq + 2 * hkv), static_cast<unsigned>(m)),
                     dim3(d / 2), 0, st, q, k, v, hq, hkv, d, m, p0, max_len, std::log2(static_cast<double>(theta)),
                     interleaved, q_out, kc, vc, q_gain, k_gain, eps, reinterpret_cast<const float2*>(table));
  return hipGetLastError();
}

hipError_t launch_heads_to_rows(const float* o, int32_t h, int64_t m, int32_t d, uint16_t* out, hipStream_t st) {
  hipLaunchKernelGGL(heads_to_rows_kernel, dim3(spread_blocks(static_cast<int64_t>(h) * m * d)), dim3(256), 0, st, o,
                     h, m, d, out);
  return hipGetLastError();
}

hipError_t launch_swiglu(const float* g, const float* u, int64_t n, uint16_t* out, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_kernel, dim3(spread_blocks(n)), dim3(256), 0, st, g, u, n, out);
  return hipGetLastError();
}

hipError_t launch_cast_f16(const float* x, int64_t n, uint16_t* y, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(cast_f16_kernel, dim3(spread_blocks(n)), dim3(256), 0, st, x, n, y);
  return hipGetLastError();
}

hipError_t launch_argmax(const float* x, int64_t n, int32_t* token, void* ws, hipStream_t st) {
  const int64_t want = (n + 4095) / 4096;
  const int nb = static_cast<int>(want < kArgmaxBlocks ? want : kArgmaxBlocks);
  float* pv = static_cast<float*>(ws);
  int32_t* pi = reinterpret_cast<int32_t*>(pv + kArgmaxBlocks);
  hipLaunchKernelGGL(argmax_partial_kernel, dim3(nb), dim3(256), 0, st, x, n, pv, pi, token);
  if (nb == 1) return hipGetLastError();
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(argmax_final_kernel, dim3(1), dim3(256), 0, st, pv, pi, nb, token);
  return hipGetLastError();
}

}  // namespace qm
