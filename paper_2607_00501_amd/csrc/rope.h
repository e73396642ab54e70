// Rotary position embedding of one pair (BaseRT Sec. 3.2: the RoPE kernel),
// shared by the standalone RoPE + cache-append kernel and the decode
// attention that folds it in, so both give the same bits: element i pairs
// with i + D/2, angle pos * theta^(-2i/D) in fp64, its sine and cosine
// rounded to fp32, the rotation in fp32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qm {

// Returns (cos, sin) in registers.
__device__ __forceinline__ float2 rope_cos_sin(int64_t pos, int i, int d, double log2_theta) {
#pragma clang fp contract(off)
  const double ang = static_cast<double>(pos) * exp2(-2.0 * i / d * log2_theta);
  return make_float2(static_cast<float>(cos(ang)), static_cast<float>(sin(ang)));
}

// Frequency of pair i under the Llama 3 long-context rule, fp64: the plain
// frequency f = theta^(-2i/D) is kept while its wavelength w = 2 pi / f is
// below orig / high, divided by factor once w exceeds orig / low, and in
// between blended as (1 - t) f / factor + t f with
// t = (orig / w - low) / (high - low), which is linear in orig / w and meets
// both outer rules at the band's edges.
__device__ __forceinline__ double rope_freq_llama3(int i, int d, double log2_theta, double factor, double low,
                                                   double high, double orig) {
#pragma clang fp contract(off)
  const double f = exp2(-2.0 * i / d * log2_theta);
  const double w = 2.0 * 3.14159265358979323846 / f;
  if (w < orig / high) return f;
  if (w > orig / low) return f / factor;
  const double t = (orig / w - low) / (high - low);
  return (1.0 - t) * f / factor + t * f;
}

// (a, b) = (x[i], x[i + D/2]) -> the rotated x[i] and x[i + D/2].  The
// fused multiply-adds are explicit and the compiler may not contract the
// remaining product into anything else, so every kernel rounds alike.
__device__ __forceinline__ float rope_low(float a, float b, float c, float s) {
#pragma clang fp contract(off)
  return fmaf(a, c, -(b * s));
}
__device__ __forceinline__ float rope_high(float a, float b, float c, float s) {
#pragma clang fp contract(off)
  return fmaf(b, c, a * s);
}

}  // namespace qm
