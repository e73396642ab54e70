// Decode attention over a pre-allocated KV cache (BaseRT Sec. 3.2: the KV
// cache is allocated to the maximum context length at load time, in a layout
// chosen for coalesced access during attention; Sec. 3.3: attention is one of
// the paths whose operator sequence is fused).
//
// One decode step of grouped-query attention: query head h reads KV head
// g = h / G (G = Hq / Hkv) and computes o_h = softmax(scale * K_g q_h) V_g over
// the first `len` rows of the cache.  Mapping on gfx950 (split-K over the
// cache length, "flash decoding"):
//  * the cache is [Hkv][max_len][D] fp16, rows of D contiguous halves, so a
//    row is 128 or 256 contiguous bytes and D/8 lanes load it with one
//    16-byte load each (fully coalesced, 4 or 8 rows per wavefront load);
//  * workgroup (split, g) takes a slice of rows of KV head g for all G query
//    heads of the group, so each K and V byte is read once per step;
//  * scores: per lane a partial dot product of its 8 dimensions
//    (v_dot2_f32_f16 against the query slice held in registers), summed over
//    the row's lanes with cross-lane adds, scaled into the base-2 domain and
//    kept in LDS; then per head the slice maximum, p = 2^(s - m) and their
//    sum; then acc = sum_t p_t v_t in fp32 registers, summed over lanes and
//    wavefronts;
//  * each workgroup writes (acc, m, l) of its slice to the caller's
//    workspace, and a second kernel merges the slices exactly as online
//    softmax does: M = max m_i, L = sum l_i 2^(m_i - M), o = sum acc_i
//    2^(m_i - M) / L.
#include "qm_internal.h"

#include <hip/hip_fp16.h>

#include <algorithm>

namespace qm {
namespace {

constexpr int kAttnWaves = 4;
constexpr int kAttnUnroll = 4;    // row loads in flight per lane

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

template <int D, int G>
__global__ __launch_bounds__(kAttnWaves * 64) void attn_decode_split_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    int64_t len, int64_t max_len, int tc, int nsplit, float scale_log2, float* __restrict__ ws) {
  constexpr int LPR = D / 8;                 // lanes per cache row
  constexpr int RPW = 64 / LPR;              // rows per wavefront load
  constexpr int RPI = kAttnWaves * RPW;      // rows per workgroup load
  extern __shared__ float sc[];              // [G][tc] scores, then p
  __shared__ float stat[G][2];               // per head: slice maximum (base 2) and sum of p
  __shared__ float part[kAttnWaves][G][D];

  const int split = blockIdx.x, g = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane % LPR, rw = lane / LPR;
  const int64_t t0 = static_cast<int64_t>(split) * tc;
  const int nrows = static_cast<int>(min<int64_t>(tc, len - t0));

  // Query slices of the G heads: dimensions 8 sub .. 8 sub + 7.
  half2v qf[G][4];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const uint4 t = *reinterpret_cast<const uint4*>(q + (static_cast<int64_t>(g) * G + j) * D + sub * 8);
    qf[j][0] = __builtin_bit_cast(half2v, t.x); qf[j][1] = __builtin_bit_cast(half2v, t.y);
    qf[j][2] = __builtin_bit_cast(half2v, t.z); qf[j][3] = __builtin_bit_cast(half2v, t.w);
  }
  const int64_t head_row0 = static_cast<int64_t>(g) * max_len + t0;
  const uint16_t* kb = k + head_row0 * D + sub * 8;
  const uint16_t* vb = v + head_row0 * D + sub * 8;

  // Scores, kAttnUnroll row loads in flight per lane (rows past the slice
  // re-read its last row and are not stored).  The V rows of the first block
  // are loaded together with its K rows, so that a slice of one block costs
  // one memory round trip.
  uint4 vpre[kAttnUnroll];
  for (int r0 = 0; r0 < nrows; r0 += RPI * kAttnUnroll) {
    uint4 kv[kAttnUnroll];
#pragma unroll
    for (int u = 0; u < kAttnUnroll; ++u) {
      const int r = min(r0 + u * RPI + wave * RPW + rw, nrows - 1);
      kv[u] = *reinterpret_cast<const uint4*>(kb + static_cast<int64_t>(r) * D);
    }
    if (r0 == 0) {
#pragma unroll
      for (int u = 0; u < kAttnUnroll; ++u) {
        const int r = min(u * RPI + wave * RPW + rw, nrows - 1);
        vpre[u] = *reinterpret_cast<const uint4*>(vb + static_cast<int64_t>(r) * D);
      }
    }
#pragma unroll
    for (int u = 0; u < kAttnUnroll; ++u) {
      const int r = r0 + u * RPI + wave * RPW + rw;
      float s[G];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        float a = __builtin_amdgcn_fdot2(qf[j][0], __builtin_bit_cast(half2v, kv[u].x), 0.0f, false);
        a = __builtin_amdgcn_fdot2(qf[j][1], __builtin_bit_cast(half2v, kv[u].y), a, false);
        a = __builtin_amdgcn_fdot2(qf[j][2], __builtin_bit_cast(half2v, kv[u].z), a, false);
        a = __builtin_amdgcn_fdot2(qf[j][3], __builtin_bit_cast(half2v, kv[u].w), a, false);
#pragma unroll
        for (int off = 1; off < LPR; off <<= 1) a += __shfl_xor(a, off);
        s[j] = a;
      }
      if (sub == 0 && r < nrows) {
#pragma unroll
        for (int j = 0; j < G; ++j) sc[j * tc + r] = s[j] * scale_log2;
      }
    }
  }
  __syncthreads();

  // Per head: slice maximum, p = 2^(s - m), sum of p.
  for (int j = wave; j < G; j += kAttnWaves) {
    float m = -INFINITY;
    for (int t = lane; t < nrows; t += 64) m = fmaxf(m, sc[j * tc + t]);
    m = wave_max(m);
    float l = 0.0f;
    for (int t = lane; t < nrows; t += 64) {
      const float p = exp2f(sc[j * tc + t] - m);
      sc[j * tc + t] = p;
      l += p;
    }
    l = wave_sum(l);
    if (lane == 0) { stat[j][0] = m; stat[j][1] = l; }
  }
  __syncthreads();

  // acc = sum_t p_t v_t over the slice.
  float acc[G][8];
#pragma unroll
  for (int j = 0; j < G; ++j)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[j][i] = 0.0f;
  for (int r0 = 0; r0 < nrows; r0 += RPI * kAttnUnroll) {
    uint4 vv[kAttnUnroll];
#pragma unroll
    for (int u = 0; u < kAttnUnroll; ++u) {
      const int r = min(r0 + u * RPI + wave * RPW + rw, nrows - 1);
      vv[u] = r0 == 0 ? vpre[u] : *reinterpret_cast<const uint4*>(vb + static_cast<int64_t>(r) * D);
    }
#pragma unroll
    for (int u = 0; u < kAttnUnroll; ++u) {
      const int r = r0 + u * RPI + wave * RPW + rw;
      const bool ok = r < nrows;
      const int rc = ok ? r : nrows - 1;
      const uint32_t w[4] = {vv[u].x, vv[u].y, vv[u].z, vv[u].w};
      float vf[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const half2v h = __builtin_bit_cast(half2v, w[i]);
        vf[2 * i] = static_cast<float>(h[0]);
        vf[2 * i + 1] = static_cast<float>(h[1]);
      }
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float p = ok ? sc[j * tc + rc] : 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[j][i] = fmaf(p, vf[i], acc[j][i]);
      }
    }
  }
  // Lanes with the same dimension slice (equal sub) hold different rows.
#pragma unroll
  for (int j = 0; j < G; ++j)
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int off = LPR; off < 64; off <<= 1) acc[j][i] += __shfl_xor(acc[j][i], off);
  if (rw == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int i = 0; i < 8; ++i) part[wave][j][sub * 8 + i] = acc[j][i];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < G * D; e += kAttnWaves * 64) {
    const int j = e / D, d = e % D;
    float a = part[0][j][d];
#pragma unroll
    for (int w2 = 1; w2 < kAttnWaves; ++w2) a += part[w2][j][d];
    ws[((static_cast<int64_t>(g) * G + j) * nsplit + split) * (D + 2) + d] = a;
  }
  if (threadIdx.x < G) {
    float* st = ws + ((static_cast<int64_t>(g) * G + threadIdx.x) * nsplit + split) * (D + 2) + D;
    st[0] = stat[threadIdx.x][0];
    st[1] = stat[threadIdx.x][1];
  }
}

// Merge of the slices of one query head (thread d: output dimension d).
// The slice statistics go to LDS in one round of loads; the partial sums of
// all slices are then loaded independently of each other (eight in flight
// per thread), so the merge costs a few memory round trips, not one per
// slice.
template <int D>
__global__ __launch_bounds__(D) void attn_decode_combine_kernel(const float* __restrict__ ws, int nsplit,
                                                                 float* __restrict__ o) {
  __shared__ float wt[kAttnMaxSplits];
  __shared__ float red[2][D / 64];
  const int h = blockIdx.x, d = threadIdx.x, lane = d & 63, wv = d >> 6;
  const float* base = ws + static_cast<int64_t>(h) * nsplit * (D + 2);
  float mloc = -INFINITY;
  float lv[kAttnMaxSplits / D];
#pragma unroll
  for (int u = 0; u < kAttnMaxSplits / D; ++u) {
    const int i = d + u * D;
    const float m = i < nsplit ? base[i * (D + 2) + D] : -INFINITY;
    lv[u] = i < nsplit ? base[i * (D + 2) + D + 1] : 0.0f;
    if (i < nsplit) wt[i] = m;
    mloc = fmaxf(mloc, m);
  }
  mloc = wave_max(mloc);
  if (lane == 0) red[0][wv] = mloc;
  __syncthreads();
  float M = red[0][0];
#pragma unroll
  for (int w2 = 1; w2 < D / 64; ++w2) M = fmaxf(M, red[0][w2]);
  float lpart = 0.0f;
#pragma unroll
  for (int u = 0; u < kAttnMaxSplits / D; ++u) {
    const int i = d + u * D;
    if (i < nsplit) {
      const float e = exp2f(wt[i] - M);
      wt[i] = e;
      lpart = fmaf(e, lv[u], lpart);
    }
  }
  lpart = wave_sum(lpart);
  if (lane == 0) red[1][wv] = lpart;
  __syncthreads();
  float L = red[1][0];
#pragma unroll
  for (int w2 = 1; w2 < D / 64; ++w2) L += red[1][w2];
  float a = 0.0f;
#pragma unroll 8
  for (int i = 0; i < nsplit; ++i) a = fmaf(wt[i], base[i * (D + 2) + d], a);
  o[static_cast<int64_t>(h) * D + d] = a / L;
}

template <int D, int G>
hipError_t launch_decode_dg(const uint16_t* q, const uint16_t* k, const uint16_t* v, int hkv, int64_t len,
                            int64_t max_len, float scale, float* o, float* ws, const AttnPlan& p, hipStream_t st) {
  const size_t lds = static_cast<size_t>(G) * p.tc * sizeof(float);
  hipLaunchKernelGGL((attn_decode_split_kernel<D, G>), dim3(p.nsplit, hkv), dim3(kAttnWaves * 64), lds, st, q, k, v,
                     len, max_len, p.tc, p.nsplit, scale * 1.4426950408889634f, ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_decode_combine_kernel<D>), dim3(hkv * G), dim3(D), 0, st, ws, p.nsplit, o);
  return hipGetLastError();
}

template <int D>
hipError_t launch_decode_d(int group, const uint16_t* q, const uint16_t* k, const uint16_t* v, int hkv, int64_t len,
                           int64_t max_len, float scale, float* o, float* ws, const AttnPlan& p, hipStream_t st) {
  switch (group) {
    case 1: return launch_decode_dg<D, 1>(q, k, v, hkv, len, max_len, scale, o, ws, p, st);
    case 2: return launch_decode_dg<D, 2>(q, k, v, hkv, len, max_len, scale, o, ws, p, st);
    case 3: return launch_decode_dg<D, 3>(q, k, v, hkv, len, max_len, scale, o, ws, p, st);
    case 4: return launch_decode_dg<D, 4>(q, k, v, hkv, len, max_len, scale, o, ws, p, st);
    case 5: return launch_decode_dg<D, 5>(q, k, v, hkv, len, max_len, scale, o, ws, p, st);
    case 6: return launch_decode_dg<D, 6>(q, k, v, hkv, len, max_len, scale, o, ws, p, st);
    case 7: return launch_decode_dg<D, 7>(q, k, v, hkv, len, max_len, scale, o, ws, p, st);
    default: return launch_decode_dg<D, 8>(q, k, v, hkv, len, max_len, scale, o, ws, p, st);
  }
}

}  // namespace

// Slices: enough workgroups for about two per CU over the KV heads, at
// least 32 rows each (a multiple of 32), at most kAttnMaxSplits slices, and
// few enough rows that the G x rows scores fit in 32 KiB of LDS.
AttnPlan attn_decode_plan(int hkv, int group, int64_t len, int cu_count) {
  const int64_t want = (2 * static_cast<int64_t>(cu_count) + hkv - 1) / hkv;
  const int64_t tc_max = kAttnScoreFloats / group / 32 * 32;
  int64_t nsplit = std::min<int64_t>(std::min<int64_t>(want, kAttnMaxSplits), (len + 31) / 32);
  nsplit = std::max<int64_t>(nsplit, (len + tc_max - 1) / tc_max);
  nsplit = std::max<int64_t>(nsplit, 1);
  int64_t tc = (len + nsplit - 1) / nsplit;
  tc = (tc + 31) / 32 * 32;
  nsplit = (len + tc - 1) / tc;
  return AttnPlan{static_cast<int>(tc), static_cast<int>(nsplit)};
}

size_t attn_decode_workspace_bytes(int32_t hq, int32_t d) {
  return static_cast<size_t>(hq) * kAttnMaxSplits * (d + 2) * sizeof(float);
}

hipError_t launch_attn_decode(const uint16_t* q, const uint16_t* k, const uint16_t* v, int32_t hq, int32_t hkv,
                              int32_t d, int64_t len, int64_t max_len, float scale, float* o, float* ws,
                              int cu_count, hipStream_t st) {
  const int group = hq / hkv;
  const AttnPlan p = attn_decode_plan(hkv, group, len, cu_count);
  return d == 64 ? launch_decode_d<64>(group, q, k, v, hkv, len, max_len, scale, o, ws, p, st)
                 : launch_decode_d<128>(group, q, k, v, hkv, len, max_len, scale, o, ws, p, st);
}

}  // namespace qm
