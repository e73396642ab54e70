// Decode attention over a pre-allocated KV cache (BaseRT Sec. 3.2: the cache
// is sized for the longest context when the model loads, and its layout is
// picked so that attention reads it coalesced; Sec. 3.3: attention is one of
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
#include <cfloat>
#include <cmath>

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

// Output element i: fp32 into o, or, when o16 is set, fp16 (round to
// nearest even) into o16.
__device__ __forceinline__ void store_out(float* o, uint16_t* o16, int64_t i, float v) {
  if (o16) {
    const _Float16 h = static_cast<_Float16>(v);
    o16[i] = __builtin_bit_cast(uint16_t, h);
  } else {
    o[i] = v;
  }
}

template <int D, int G>
__global__ __launch_bounds__(kAttnWaves * 64) void attn_decode_split_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    int64_t len, int64_t max_len, int tc, int nsplit, float scale_log2, float* __restrict__ ws,
    float* __restrict__ o, uint16_t* __restrict__ o16) {
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
  if (o || o16) {   // a single slice covers the whole cache: normalise and write the output
    for (int e = threadIdx.x; e < G * D; e += kAttnWaves * 64) {
      const int j = e / D, d = e % D;
      float a = part[0][j][d];
#pragma unroll
      for (int w2 = 1; w2 < kAttnWaves; ++w2) a += part[w2][j][d];
      store_out(o, o16, (static_cast<int64_t>(g) * G + j) * D + d, a / stat[j][1]);
    }
    return;
  }
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
                                                                 float* __restrict__ o, uint16_t* __restrict__ o16) {
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
  store_out(o, o16, static_cast<int64_t>(h) * D + d, a / L);
}

template <int D, int G>
hipError_t launch_decode_dg(const uint16_t* q, const uint16_t* k, const uint16_t* v, int hkv, int64_t len,
                            int64_t max_len, float scale, float* o, uint16_t* o16, float* ws, const AttnPlan& p,
                            hipStream_t st) {
  const size_t lds = static_cast<size_t>(G) * p.tc * sizeof(float);
  const float sl2 = scale * 1.4426950408889634f;
  float* od = p.nsplit == 1 ? o : nullptr;
  uint16_t* od16 = p.nsplit == 1 ? o16 : nullptr;
  hipLaunchKernelGGL((attn_decode_split_kernel<D, G>), dim3(p.nsplit, hkv), dim3(kAttnWaves * 64), lds, st,
                     q, k, v, len, max_len, p.tc, p.nsplit, sl2, ws, od, od16);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.nsplit == 1) return e;
  hipLaunchKernelGGL((attn_decode_combine_kernel<D>), dim3(hkv * G), dim3(D), 0, st, ws, p.nsplit, o, o16);
  return hipGetLastError();
}

template <int D>
hipError_t launch_decode_d(int group, const uint16_t* q, const uint16_t* k, const uint16_t* v, int hkv, int64_t len,
                           int64_t max_len, float scale, float* o, uint16_t* o16, float* ws, const AttnPlan& p,
                           hipStream_t st) {
  switch (group) {
    case 1: return launch_decode_dg<D, 1>(q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
    case 2: return launch_decode_dg<D, 2>(q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
    case 3: return launch_decode_dg<D, 3>(q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
    case 4: return launch_decode_dg<D, 4>(q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
    case 5: return launch_decode_dg<D, 5>(q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
    case 6: return launch_decode_dg<D, 6>(q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
    case 7: return launch_decode_dg<D, 7>(q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
    default: return launch_decode_dg<D, 8>(q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
  }
}

// ------------------------------------------------------------------ prefill

typedef _Float16 half4v __attribute__((ext_vector_type(4)));

// Causal FlashAttention for a prompt chunk (Sec. 3.4: attention over key
// tiles, each query row carrying its running maximum and sum, memory linear
// in the length).  Workgroup = one
// query head x 128 query rows, four wavefronts of 32 rows.  Per block of 64
// keys (32 for head_dim 128, to fit 256 VGPRs; K row-major and V transposed
// in LDS, the next blocks loading into registers meanwhile), each wavefront
// computes S^T = K Q^T as independent 32-key tiles with v_mfma_f32_32x32x16_f16 (lane l then holds 32
// keys of query l%32, so the row statistics need one cross-lane step), masks
// future positions on the diagonal blocks, updates the running maximum and
// sum in the base-2 domain, rescales its O^T accumulators when the maximum
// moved and adds V^T P^T.  The k slots of that second product are relabelled
// to the keys the lane already holds, so P never leaves its lane.
template <int D>
__global__ __launch_bounds__(256, 3) void attn_prefill_kernel(const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v, int group,
                                                           int64_t m, int64_t p0, int64_t max_len, float scale_log2,
                                                           float* __restrict__ o, int n_heads, int cu_count, int bmax,
                                                           int64_t n_units, float* __restrict__ ws,
                                                           uint16_t* __restrict__ o16) {
  constexpr int KB = D == 64 ? 64 : 32;      // keys per block (head_dim 128: 32, to fit 256 VGPRs)
  constexpr int NT = KB / 32;                // 32-key S tiles per block
  constexpr int KS = D / 16;                 // k steps of S over the head dimension
  constexpr int DB = D / 32;                 // 32-wide blocks of the head dimension
  constexpr int KPAD = D + 8;                // LDS row of K (halves)
  constexpr int VPAD = KB + 4;               // LDS row of V^T (halves): an even number of dwords, 2 mod 4
  constexpr int CHUNKS = KB * D / 8;         // 16-byte pieces of a block
  constexpr int PER_T = CHUNKS / 256;        // pieces per thread
  __shared__ __attribute__((aligned(16))) _Float16 ks[KB * KPAD];
  __shared__ __attribute__((aligned(16))) _Float16 vt[D * VPAD];

  // Units (tile, key split, head), tiles in order of decreasing causal
  // length (longest first); a tile of nb key blocks is split into
  // ceil(nb / bmax) ranges of at most bmax blocks.  Workgroup L is dealt to a
  // CU in round L / cu_count, and the rounds share the CUs in the same order,
  // so every second round is dealt in reverse: the CU that took one of the
  // longest units also takes one of the shortest (a partial last round keeps
  // its order where reversal would leave it).  Measured: 512 workgroups of
  // Llama-3.2-1B at m = 2048 took 52 -> 42 us.
  // Positions and key counts fit 32 bits (max_len <= 262144, m <= 65536;
  // units < 2^31), which keeps them out of 64-bit register pairs.
  const int ntiles = static_cast<int>((m + 127) / 128);
  const int mi = static_cast<int>(m), p0i = static_cast<int>(p0);
  const int L = static_cast<int>(blockIdx.x);
  const int rnd = L / cu_count, pos = L % cu_count;
  const int rev = rnd * cu_count + (cu_count - 1 - pos);
  const int u = (rnd & 1) && rev < n_units ? rev : L;
  int tile = ntiles - 1, nsplit = 1, cum = 0, slot = 0;           // units / split slots before the tile
  for (; tile > 0; --tile) {
    const int nb = (p0i + min(128 * (tile + 1), mi) + KB - 1) / KB;
    nsplit = (nb + bmax - 1) / bmax;
    const int nu = nsplit * n_heads;
    if (u < cum + nu) break;
    cum += nu;
    slot += nsplit > 1 ? nsplit : 0;
  }
  if (tile == 0) nsplit = ((p0i + min(128, mi) + KB - 1) / KB + bmax - 1) / bmax;
  const int split = (u - cum) / n_heads;
  const int h = (u - cum) % n_heads, g = h / group;
  // Row records of this unit's partial (split tiles only; 128 rows of D + 4
  // floats: unnormalised sums, maximum, denominator, 2 pad).
  float* const part =
      nsplit > 1 ? ws + (static_cast<int64_t>(slot + split) * n_heads + h) * 128 * (D + 4) : nullptr;
  const int lane = threadIdx.x & 63, lh = lane >> 5, col = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q0 = tile * 128;
  const int qrow = q0 + 32 * wave + col;                          // this lane's query row
  const int qpos = p0i + min(qrow, mi - 1);                       // its position
  const int nkeys = p0i + min(q0 + 128, mi);                      // keys of the tile
  const int kb_lo = split * bmax * KB;                            // this unit's key range
  const int kb_hi = min(nkeys, kb_lo + bmax * KB);
  const int wave_first = p0i + q0 + 32 * wave;                    // first query position of the wavefront
  const int wave_last = p0i + min(q0 + 32 * wave + 31, mi - 1);

  // Q fragments (B operand of S^T = K Q^T): query col, dims 16 s + 8 lh + 0..7.
  half8v qf[KS];
  const uint16_t* qr = q + (static_cast<int64_t>(h) * m + min(qrow, mi - 1)) * D;
#pragma unroll
  for (int s = 0; s < KS; ++s) qf[s] = *reinterpret_cast<const half8v*>(qr + 16 * s + 8 * lh);

  const uint16_t* kh = k + static_cast<int64_t>(g) * max_len * D;
  const uint16_t* vh = v + static_cast<int64_t>(g) * max_len * D;
  // K pieces row-major (consecutive threads along a row); V in pairs of
  // keys (consecutive threads on consecutive key pairs of one 8-dimension
  // chunk), so that each transposed LDS write of a wavefront is a dword of
  // two keys and the writes of a wavefront fill consecutive dwords of V^T
  // rows.
  // Blocks past the end load clamped (valid) rows and are never used, so
  // the loads carry no branch and the register sets stay in registers.
  struct Blk { uint4 k[PER_T], v[PER_T]; };
  auto load_block = [&](int kb0) __attribute__((always_inline)) {
    Blk b;
#pragma unroll
    for (int c = 0; c < PER_T; ++c) {
      const int piece = threadIdx.x + 256 * c;
      const int row = piece / (D / 8), off = (piece % (D / 8)) * 8;
      b.k[c] = *reinterpret_cast<const uint4*>(kh + min(kb0 + row, nkeys - 1) * D + off);
    }
#pragma unroll
    for (int c = 0; c < PER_T / 2; ++c) {
      const int pp = threadIdx.x + 256 * c;                      // a pair of keys, 8 dimensions
      const int kp = pp % (KB / 2), voff = (pp / (KB / 2)) * 8;
      b.v[2 * c] = *reinterpret_cast<const uint4*>(vh + min(kb0 + 2 * kp, nkeys - 1) * D + voff);
      b.v[2 * c + 1] = *reinterpret_cast<const uint4*>(vh + min(kb0 + 2 * kp + 1, nkeys - 1) * D + voff);
    }
    return b;
  };
  auto store_block = [&](const Blk& b) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < PER_T; ++c) {
      const int piece = threadIdx.x + 256 * c;
      const int row = piece / (D / 8), off = (piece % (D / 8)) * 8;
      *reinterpret_cast<uint4*>(&ks[row * KPAD + off]) = b.k[c];
    }
    // V^T: dimension d of keys 2 kp, 2 kp + 1 as one dword.
#pragma unroll
    for (int c = 0; c < PER_T / 2; ++c) {
      const int pp = threadIdx.x + 256 * c;
      const int kp = pp % (KB / 2), voff = (pp / (KB / 2)) * 8;
      const uint32_t w0[4] = {b.v[2 * c].x, b.v[2 * c].y, b.v[2 * c].z, b.v[2 * c].w};
      const uint32_t w1[4] = {b.v[2 * c + 1].x, b.v[2 * c + 1].y, b.v[2 * c + 1].z, b.v[2 * c + 1].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *reinterpret_cast<uint32_t*>(&vt[(voff + 2 * i) * VPAD + 2 * kp]) = __builtin_amdgcn_perm(w1[i], w0[i], 0x05040100u);
        *reinterpret_cast<uint32_t*>(&vt[(voff + 2 * i + 1) * VPAD + 2 * kp]) =
            __builtin_amdgcn_perm(w1[i], w0[i], 0x07060302u);
      }
    }
  };

  float16v acc[DB];
#pragma unroll
  for (int b = 0; b < DB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = 0.0f;
  float m_run = -FLT_MAX, l_run = 0.0f;

  auto compute = [&](int kb0) __attribute__((always_inline)) {
    if (kb0 <= wave_last) {
      // S^T for keys kb0 + 32 t + (lane's rows), query col: two independent tiles.
      float16v st[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) st[t][r] = 0.0f;
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const half8v a = *reinterpret_cast<const half8v*>(&ks[(32 * t + col) * KPAD + 16 * s + 8 * lh]);
          st[t] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, qf[s], st[t], 0, 0, 0);
        }
      // Causal mask only where the block reaches past the wavefront's first
      // query, on 32-bit offsets inside the block; the maximum is taken on
      // the raw scores (scale > 0) and scaled once.
      float bm = -INFINITY;
      if (kb0 + KB - 1 > wave_first) {
        const int lim = min(qpos - kb0, KB) - 4 * lh;              // >= 0: key offset allowed
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float x = 32 * t + 8 * (r >> 2) + (r & 3) <= lim ? st[t][r] : -INFINITY;
            st[t][r] = x;
            bm = fmaxf(bm, x);
          }
      } else {
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) bm = fmaxf(bm, st[t][r]);
      }
      bm = fmaxf(bm, __shfl_xor(bm, 32)) * scale_log2;
      // m_run starts at -FLT_MAX, not -inf: a row with no key yet in this
      // unit's range (a later key split) keeps a finite maximum, so its p and
      // alpha come out 0 instead of NaN; other rows are unchanged.
      const float m_new = fmaxf(m_run, bm);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);   // v_exp_f32 (0 on the first block)
      float rs = 0.0f;
      half8v pf[2 * NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float p0v = __builtin_amdgcn_exp2f(fmaf(st[t][r], scale_log2, -m_new));
          const float p1v = __builtin_amdgcn_exp2f(fmaf(st[t][r + 1], scale_log2, -m_new));
          rs += p0v + p1v;
          const half2v pp = __builtin_bit_cast(half2v, __builtin_amdgcn_cvt_pkrtz(p0v, p1v));
          pf[2 * t + (r >> 3)][r & 7] = pp[0];
          pf[2 * t + (r >> 3)][(r & 7) + 1] = pp[1];
        }
      rs += __shfl_xor(rs, 32);
      l_run = fmaf(l_run, alpha, rs);
      m_run = m_new;
      if (__builtin_amdgcn_ballot_w64(alpha != 1.0f) != 0) {         // the running maximum moved
#pragma unroll
        for (int b = 0; b < DB; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[b][r] *= alpha;
      }
      // O^T += V^T P^T; k slot (lh, i) of step kk is key 16 kk + 8 (i / 4) + 4 lh + i % 4.
#pragma unroll
      for (int kk = 0; kk < KB / 16; ++kk)
#pragma unroll
        for (int b = 0; b < DB; ++b) {
          const _Float16* vrow = &vt[(32 * b + col) * VPAD + 16 * kk + 4 * lh];
          const half4v lo = *reinterpret_cast<const half4v*>(vrow);
          const half4v hi = *reinterpret_cast<const half4v*>(vrow + 8);
          const half8v a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, pf[kk], acc[b], 0, 0, 0);
        }
    }
  };

  // Register sets of block loads: the loads of block b + 2 (head_dim 64) or
  // b + 1 (head_dim 128) are issued right after block b has gone to LDS, so
  // they land during the math.
  if constexpr (D == 64) {
    Blk b0 = load_block(kb_lo), b1 = load_block(kb_lo + KB);
    for (int kb0 = kb_lo; kb0 < kb_hi; kb0 += 2 * KB) {
      store_block(b0);
      __syncthreads();
      b0 = load_block(kb0 + 2 * KB);
      compute(kb0);
      __syncthreads();
      if (kb0 + KB < kb_hi) {
        store_block(b1);
        __syncthreads();
        b1 = load_block(kb0 + 3 * KB);
        compute(kb0 + KB);
        __syncthreads();
      }
    }
  } else {
    // head_dim 128: one register set (two would not fit in 256 VGPRs).
    Blk b0 = load_block(kb_lo);
    for (int kb0 = kb_lo; kb0 < kb_hi; kb0 += KB) {
      store_block(b0);
      __syncthreads();
      b0 = load_block(kb0 + KB);
      compute(kb0);
      __syncthreads();
    }
  }
  if (qrow < mi) {
    if (!part && o16) {
      // fp16 rows [m][n_heads * D] (the output projection's input): the four
      // consecutive dimensions of r = 4j .. 4j + 3 as one 8-byte store.
      const float inv = 1.0f / l_run;
      uint16_t* orow = o16 + (static_cast<int64_t>(qrow) * n_heads + h) * D;
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const half2v lo = {static_cast<_Float16>(acc[b][4 * j] * inv), static_cast<_Float16>(acc[b][4 * j + 1] * inv)};
          const half2v hi = {static_cast<_Float16>(acc[b][4 * j + 2] * inv),
                             static_cast<_Float16>(acc[b][4 * j + 3] * inv)};
          *reinterpret_cast<uint2*>(orow + 32 * b + 8 * j + 4 * lh) =
              make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
        }
    } else if (!part) {
      const float inv = 1.0f / l_run;
      float* orow = o + (static_cast<int64_t>(h) * m + qrow) * D;
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) orow[32 * b + 8 * (r >> 2) + 4 * lh + (r & 3)] = acc[b][r] * inv;
    } else {
      // Partial of this key range: unnormalised sums, running maximum (base
      // 2) and sum, in a row record of D + 4 floats (16-byte aligned), merged
      // by attn_prefill_merge_kernel.
      float* prow = part + (qrow - q0) * (D + 4);
#pragma unroll
      for (int b = 0; b < DB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) prow[32 * b + 8 * (r >> 2) + 4 * lh + (r & 3)] = acc[b][r];
      if (lh == 0) {
        prow[D] = m_run;
        prow[D + 1] = l_run;
      }
    }
  }
}

// Merge of the key splits of the split tiles: for each row, M = max of the
// splits' maxima, L = sum of l_s 2^(m_s - M), o = sum of acc_s 2^(m_s - M) / L,
// the splits taken in order (in batches, each rescaling the sums so far to
// the batch's new maximum).  Workgroup = (split tile, head, group of
// 256 / (D/4) rows); thread = (row, 4 dimensions); the loads of kMergeBatch
// splits are issued before their use.
constexpr int kMergeBatch = 8;

template <int D>
__global__ __launch_bounds__(256) void attn_prefill_merge_kernel(const float* __restrict__ ws, int64_t m, int64_t p0,
                                                                 int n_heads, int bmax, float* __restrict__ o,
                                                                 uint16_t* __restrict__ o16) {
  constexpr int KB = D == 64 ? 64 : 32;
  constexpr int C4 = D / 4;                                       // threads per row
  constexpr int RW = 256 / C4;                                    // rows per workgroup
  constexpr int GROUPS = 128 / RW;
  const int ntiles = static_cast<int>((m + 127) / 128);
  const int gi = static_cast<int>(blockIdx.x % GROUPS);
  const int rest = static_cast<int>(blockIdx.x / GROUPS);
  const int c = rest / n_heads, h = rest % n_heads;
  int tile = ntiles - 1, nsplit = 1, seen = 0;
  int64_t slot = 0;
  for (; tile >= 0; --tile) {
    const int64_t nb = (p0 + min<int64_t>(128 * (tile + 1), m) + KB - 1) / KB;
    nsplit = static_cast<int>((nb + bmax - 1) / bmax);
    if (nsplit > 1) {
      if (seen == c) break;
      ++seen;
      slot += nsplit;
    }
  }
  if (tile < 0) return;                                           // (never: the grid counts split tiles)
  const int rows = static_cast<int>(min<int64_t>(128, m - 128 * static_cast<int64_t>(tile)));
  const int r = gi * RW + static_cast<int>(threadIdx.x) / C4, d4 = static_cast<int>(threadIdx.x) % C4;
  if (r >= rows) return;                                          // (no barriers below)
  // Record of row r in split sp: D sums, maximum, denominator, 2 pad floats.
  auto rec = [&](int sp) { return ws + (((slot + sp) * n_heads + h) * 128 + r) * (D + 4); };
  // One pass: the running maximum moves per batch and rescales what is
  // summed so far, as online softmax does (one memory round trip per batch).
  float mx = -FLT_MAX, l = 0.0f;
  float4 a = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int s0 = 0; s0 < nsplit; s0 += kMergeBatch) {
    float mv[kMergeBatch], lv[kMergeBatch];
    float4 av[kMergeBatch];
#pragma unroll
    for (int j = 0; j < kMergeBatch; ++j) {
      const float* p = rec(min(s0 + j, nsplit - 1));
      mv[j] = p[D];
      lv[j] = p[D + 1];
      av[j] = reinterpret_cast<const float4*>(p)[d4];
    }
    float bm = mx;
#pragma unroll
    for (int j = 0; j < kMergeBatch; ++j) bm = fmaxf(bm, mv[j]);    // clamped duplicates change no maximum
    const float sc = exp2f(mx - bm);
    mx = bm;
    l *= sc;
    a.x *= sc; a.y *= sc; a.z *= sc; a.w *= sc;
#pragma unroll
    for (int j = 0; j < kMergeBatch; ++j) {
      const float w = s0 + j < nsplit ? exp2f(mv[j] - mx) : 0.0f;
      l = fmaf(lv[j], w, l);
      a.x = fmaf(w, av[j].x, a.x);
      a.y = fmaf(w, av[j].y, a.y);
      a.z = fmaf(w, av[j].z, a.z);
      a.w = fmaf(w, av[j].w, a.w);
    }
  }
  const float inv = 1.0f / l;
  const int64_t row = 128 * static_cast<int64_t>(tile) + r;
  if (o16) {
    const half2v lo = {static_cast<_Float16>(a.x * inv), static_cast<_Float16>(a.y * inv)};
    const half2v hi = {static_cast<_Float16>(a.z * inv), static_cast<_Float16>(a.w * inv)};
    reinterpret_cast<uint2*>(o16 + (row * n_heads + h) * D)[d4] =
        make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
  } else {
    reinterpret_cast<float4*>(o + (static_cast<int64_t>(h) * m + row) * D)[d4] =
        make_float4(a.x * inv, a.y * inv, a.z * inv, a.w * inv);
  }
}

}  // namespace

// Key splits of the prefill attention: the blocks of all (tile, head) units
// spread over about two workgroups per CU, at least a minimum number of
// blocks per split; then the smallest split length whose partials fit the
// workspace (the slots needed fall as the length grows; no workspace: no
// split).  Split lengths of at least 8 blocks and a longest tile of at
// least 3 lengths for head_dim 64 (64-key blocks), 4 and 2 for head_dim 128
// (32-key blocks, twice the blocks per tile and half the heads of the
// models here): fitted on MI355X over prompts of 128 .. 2048 rows from
// position 0, where finer splits lost 5-11% for head_dim 64 and gained
// 3-17% for head_dim 128.  A chunk far into the cache (a few tiles,
// thousands of key blocks each) runs on a handful of CUs without splits.
PrefillPlan attn_prefill_plan(int32_t hq, int32_t d, int64_t m, int64_t p0, int cu_count, size_t ws_bytes) {
  PrefillPlan p{};
  const int kb = d == 64 ? 64 : 32;
  const int64_t ntiles = (m + 127) / 128;
  auto blocks = [&](int64_t t) { return (p0 + std::min<int64_t>(128 * (t + 1), m) + kb - 1) / kb; };
  int64_t total = 0, longest = 0;
  for (int64_t t = 0; t < ntiles; ++t) {
    total += blocks(t);
    longest = std::max(longest, blocks(t));
  }
  total *= hq;
  const int64_t target = 2 * static_cast<int64_t>(std::max(cu_count, 1));
  const int64_t min_split = d == 64 ? 8 : 4, factor = d == 64 ? 3 : 2;
  int64_t bmax = std::max<int64_t>(min_split, (total + target - 1) / target);
  if (longest < factor * bmax) bmax = longest;          // no split
  auto slots = [&](int64_t bm) {
    int64_t sl = 0;
    for (int64_t t = 0; t < ntiles; ++t) {
      const int64_t s = (blocks(t) + bm - 1) / bm;
      sl += s > 1 ? s : 0;
    }
    return sl;
  };
  const size_t slot_bytes = static_cast<size_t>(hq) * 128 * (d + 4) * sizeof(float);
  p.ws_needed = static_cast<size_t>(slots(bmax)) * slot_bytes;
  auto fits = [&](int64_t bm) { return static_cast<size_t>(slots(bm)) * slot_bytes <= ws_bytes; };
  if (bmax >= longest || !fits(bmax)) {
    int64_t lo = bmax, hi = longest;                    // !fits(lo) or lo >= longest; fits(longest): no slots
    if (lo >= hi) {
      bmax = longest;
    } else {
      while (hi - lo > 1) {
        const int64_t mid = lo + (hi - lo) / 2;
        (fits(mid) ? hi : lo) = mid;
      }
      bmax = hi;
    }
  }
  p.bmax = static_cast<int>(std::max<int64_t>(bmax, 1));
  p.units = 0;
  p.split_tiles = 0;
  for (int64_t t = 0; t < ntiles; ++t) {
    const int64_t s = (blocks(t) + p.bmax - 1) / p.bmax;
    p.units += s * hq;
    p.split_tiles += s > 1 ? 1 : 0;
  }
  return p;
}

hipError_t launch_attn_prefill(const uint16_t* q, const uint16_t* k, const uint16_t* v, int32_t hq, int32_t hkv,
                               int32_t d, int64_t m, int64_t p0, int64_t max_len, float scale, float* o,
                               uint16_t* o16, void* ws, size_t ws_bytes, int cu_count, hipStream_t st) {
  const PrefillPlan p = attn_prefill_plan(hq, d, m, p0, cu_count, ws ? ws_bytes : 0);
  const dim3 grid(static_cast<unsigned>(p.units));
  const float sl2 = scale * 1.4426950408889634f;
  const int cu = cu_count > 0 ? cu_count : 1;
  float* wsf = static_cast<float*>(ws);
  if (d == 64)
    hipLaunchKernelGGL((attn_prefill_kernel<64>), grid, dim3(256), 0, st, q, k, v, hq / hkv, m, p0, max_len, sl2, o,
                       hq, cu, p.bmax, p.units, wsf, o16);
  else
    hipLaunchKernelGGL((attn_prefill_kernel<128>), grid, dim3(256), 0, st, q, k, v, hq / hkv, m, p0, max_len, sl2, o,
                       hq, cu, p.bmax, p.units, wsf, o16);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.split_tiles == 0) return e;
  const dim3 mg(static_cast<unsigned>(p.split_tiles * hq * (128 / (256 / (d / 4)))));
  if (d == 64)
    hipLaunchKernelGGL((attn_prefill_merge_kernel<64>), mg, dim3(256), 0, st, wsf, m, p0, hq, p.bmax, o, o16);
  else
    hipLaunchKernelGGL((attn_prefill_merge_kernel<128>), mg, dim3(256), 0, st, wsf, m, p0, hq, p.bmax, o, o16);
  return hipGetLastError();
}

// Slices: enough workgroups for about two per CU over the KV heads, at
// least 32 rows each (a multiple of 32), at most kAttnMaxSplits slices, and
// few enough rows that the G x rows scores fit in 32 KiB of LDS.
AttnPlan attn_decode_plan(int hkv, int group, int64_t len, int cu_count) {
  // Short caches: one slice per KV head, which writes the output itself (no
  // merge launch); a few memory round trips cost less than the second launch.
  if (len <= kAttnDirectLen) return AttnPlan{static_cast<int>((len + 31) / 32 * 32), 1};
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
                              int32_t d, int64_t len, int64_t max_len, float scale, float* o, uint16_t* o16,
                              float* ws, int cu_count, hipStream_t st) {
  const int group = hq / hkv;
  const AttnPlan p = attn_decode_plan(hkv, group, len, cu_count);
  return d == 64 ? launch_decode_d<64>(group, q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st)
                 : launch_decode_d<128>(group, q, k, v, hkv, len, max_len, scale, o, o16, ws, p, st);
}

}  // namespace qm
