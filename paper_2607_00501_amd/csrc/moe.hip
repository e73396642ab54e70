// Mixture-of-experts path: top-k routing, stable counting-sort bucketing,
// two grouped Q4 MFMA GEMMs (gate+up with a fused SwiGLU epilogue, then
// down with the gate weight folded in) and a deterministic combine.
//
// BaseRT runs MoE models (Sec. 4.1: Qwen3-30B-A3B, Gemma-4-26B-A4B) and
// reports its largest prefill margins there (Sec. 4.3); the kernels follow
// its fusion principle (Sec. 3.3: each fused step saves a launch and a
// global-memory round trip).  Everything is enqueued on one stream with no
// host round trip: per-expert row counts stay on the device, and each GEMM
// workgroup finds its (expert, row tile) from the counts itself.
#include <hip/hip_fp16.h>

#include "qgemm.h"

namespace qm {
namespace {

// ------------------------------------------------------------------ route

constexpr int kRouteThreads = 256;   // one wavefront per token
constexpr int kMaxPerLane = 16;      // n_experts <= 1024

__global__ __launch_bounds__(kRouteThreads) void route_kernel(const float* __restrict__ logits,
                                                              int64_t m, int E, int K,
                                                              int32_t* __restrict__ ids,
                                                              float* __restrict__ gates) {
  const int lane = threadIdx.x & 63;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * (kRouteThreads / 64) + (threadIdx.x >> 6);
  if (t >= m) return;
  const float* row = logits + t * E;
  float v[kMaxPerLane];
  const int per_lane = (E + 63) / 64;
#pragma unroll
  for (int i = 0; i < kMaxPerLane; ++i) {
    const int e = i * 64 + lane;
    v[i] = (i < per_lane && e < E) ? row[e] : -INFINITY;
  }
  uint32_t taken = 0;   // bit i: item i of this lane already selected
  float top_v[16];
  int top_e[16];
  for (int j = 0; j < K; ++j) {
    // Lane-local best: highest value, lowest expert index on ties.
    float bv = -INFINITY;
    int be = 0x7FFFFFFF;
#pragma unroll
    for (int i = 0; i < kMaxPerLane; ++i) {
      const int e = i * 64 + lane;
      if (i < per_lane && e < E && !(taken >> i & 1u)) {
        if (v[i] > bv || (v[i] == bv && e < be)) { bv = v[i]; be = e; }
      }
    }
    // Wavefront argmax with the same order.
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ov = __shfl_xor(bv, off);
      const int oe = __shfl_xor(be, off);
      if (ov > bv || (ov == bv && oe < be)) { bv = ov; be = oe; }
    }
    top_v[j] = bv;
    top_e[j] = be;
    if ((be & 63) == lane) taken |= 1u << (be >> 6);
  }
  // Softmax over the selected logits, relative to the largest.
  float denom = 0.0f;
  for (int j = 0; j < K; ++j) denom += expf(top_v[j] - top_v[0]);
  if (lane < K) {
    float val = 0.0f;
    int ex = 0;
    for (int j = 0; j < K; ++j)
      if (j == lane) { val = top_v[j]; ex = top_e[j]; }
    ids[t * K + lane] = ex;
    gates[t * K + lane] = expf(val - top_v[0]) / denom;
  }
}

// ----------------------------------------------------------------- bucket

constexpr int kBucketThreads = 1024;
constexpr int kBucketWaves = kBucketThreads / 64;

// One workgroup: histogram, exclusive scan, then a stable scatter that walks
// the assignments in order, 1024 at a time.  Inside a wavefront the lanes
// holding the same expert are found with ten ballots (one per bit of the
// expert id); their rank is the population count of the lower matching lanes,
// and lower wavefronts' counts for that expert come from LDS.
__global__ __launch_bounds__(kBucketThreads) void bucket_kernel(const int32_t* __restrict__ ids,
                                                                int64_t A, int E,
                                                                int32_t* __restrict__ counts,
                                                                int32_t* __restrict__ offsets,
                                                                int32_t* __restrict__ sorted_assign) {
  __shared__ int cnt[1024];
  __shared__ int off[1024];
  __shared__ int running[1024];
  __shared__ int wsum[kBucketWaves];
  __shared__ uint8_t wave_cnt[kBucketWaves][1024];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  cnt[tid] = 0;
  running[tid] = 0;
  for (int w = 0; w < kBucketWaves; ++w) wave_cnt[w][tid] = 0;
  __syncthreads();
  for (int64_t a = tid; a < A; a += kBucketThreads) atomicAdd(&cnt[ids[a]], 1);
  __syncthreads();
  // Exclusive scan of cnt[0..1023] (entries >= E are zero).
  {
    const int c = cnt[tid];
    int incl = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int o = __shfl_up(incl, d);
      if (lane >= d) incl += o;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += wsum[w];
    off[tid] = base + incl - c;
    __syncthreads();
    if (tid < E) {
      counts[tid] = c;
      offsets[tid] = off[tid];
    }
    if (tid == 0) offsets[E] = static_cast<int32_t>(A);
  }
  const uint64_t lower = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int64_t base = 0; base < A; base += kBucketThreads) {
    const int64_t a = base + tid;
    const bool valid = a < A;
    const int e = valid ? ids[a] : 0;
    uint64_t mask = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 10; ++bit) {
      const bool set = (e >> bit) & 1;
      const uint64_t b = __ballot(valid && set);
      mask &= set ? b : ~b;
    }
    const int rank = __popcll(mask & lower);
    const int wcount = __popcll(mask);
    const bool leader = valid && rank == 0;
    if (leader) wave_cnt[wave][e] = static_cast<uint8_t>(wcount);
    __syncthreads();
    if (valid) {
      int pre = 0;
      for (int w = 0; w < wave; ++w) pre += wave_cnt[w][e];
      sorted_assign[off[e] + running[e] + pre + rank] = static_cast<int32_t>(a);
    }
    __syncthreads();
    if (leader) {
      wave_cnt[wave][e] = 0;
      atomicAdd(&running[e], wcount);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- combine

// y[t][n] = sum over slots j (in order) of the gate-weighted expert outputs.
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ yp, float* __restrict__ y,
                                                      int64_t m, int64_t hidden, int K) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;   // float4 index
  const int64_t h4 = hidden / 4;
  if (i >= m * h4) return;
  const int64_t t = i / h4, c = i % h4;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < K; ++j) {
    const float4 v = reinterpret_cast<const float4*>(yp + (t * K + j) * hidden)[c];
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  reinterpret_cast<float4*>(y + t * hidden)[c] = s;
}

template <int BM, int WN>
hipError_t launch_moe_tiles(const MoeArgs& a, hipStream_t st) {
  const int64_t A = a.m * a.top_k;
  // Upper bound on the number of (expert, row tile) pairs: sum of
  // ceil(count_e / BM) <= A / BM + E.  Workgroups past the last tile exit.
  const unsigned tiles = static_cast<unsigned>((A + BM - 1) / BM + a.n_experts);
  QgemmArgs g{};
  g.counts = a.counts; g.offsets = a.offsets; g.sorted_assign = a.sorted_assign; g.topk_w = a.topk_w;
  g.n_experts = a.n_experts; g.top_k = a.top_k; g.M = A;
  // gate/up + SwiGLU: A = x rows gathered per assignment, N = inter, K = hidden
  g.q = a.gq; g.s = a.gs; g.q2 = a.uq; g.s2 = a.us; g.a = a.x; g.h = a.h; g.N = a.inter; g.K = a.hidden;
  const unsigned ny1 = static_cast<unsigned>((a.inter + 64 * WN - 1) / (64 * WN));
  hipLaunchKernelGGL((qgemm_kernel<BM, WN, 1, QgMode::kMoeGateUp>), dim3(tiles, ny1), dim3(WN * 64), 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // down, scaled by the gate weight and scattered to the assignment slot
  g.q = a.dq; g.s = a.ds; g.q2 = nullptr; g.s2 = nullptr; g.a = a.h; g.yp = a.yp; g.N = a.hidden; g.K = a.inter;
  const unsigned ny2 = static_cast<unsigned>((a.hidden + 64 * WN - 1) / (64 * WN));
  hipLaunchKernelGGL((qgemm_kernel<BM, WN, 1, QgMode::kMoeDown>), dim3(tiles, ny2), dim3(WN * 64), 0, st, g);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n4 = a.m * (a.hidden / 4);
  hipLaunchKernelGGL(combine_kernel, dim3(static_cast<unsigned>((n4 + 255) / 256)), dim3(256), 0, st, a.yp,
                     a.y, a.m, a.hidden, a.top_k);
  return hipGetLastError();
}

}  // namespace

size_t moe_workspace_bytes(int64_t m, int32_t top_k, int64_t hidden, int64_t inter) {
  const size_t A = static_cast<size_t>(m) * top_k;
  const size_t h_bytes = (A * inter * 2 + 255) / 256 * 256;
  const size_t yp_bytes = (A * hidden * 4 + 255) / 256 * 256;
  return h_bytes + yp_bytes;
}

const char* moe_tile_name(int64_t rows_per_expert) {
  return rows_per_expert <= 24 ? "32-row bucket tiles x 4 panels" : "64-row bucket tiles x 4 panels";
}

hipError_t launch_route(const float* logits, int64_t m, int32_t e, int32_t k, int32_t* ids, float* w,
                        int32_t* counts, int32_t* offsets, int32_t* sorted_assign, hipStream_t st) {
  if (m > 0) {
    const unsigned blocks = static_cast<unsigned>((m + 3) / 4);
    hipLaunchKernelGGL(route_kernel, dim3(blocks), dim3(kRouteThreads), 0, st, logits, m, e, k, ids, w);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(bucket_kernel, dim3(1), dim3(kBucketThreads), 0, st, ids, m * k, e, counts, offsets,
                     sorted_assign);
  return hipGetLastError();
}

hipError_t launch_moe(const MoeArgs& a, int cu_count, hipStream_t st) {
  (void)cu_count;
  // Per-chip tile choice by rows per expert: 32-row tiles when buckets are
  // small (decode-like prefill chunks), 64-row tiles otherwise.
  const int64_t rpe = a.m * a.top_k / a.n_experts;
  if (rpe <= 24) return launch_moe_tiles<32, 4>(a, st);
  return launch_moe_tiles<64, 4>(a, st);
}

}  // namespace qm
