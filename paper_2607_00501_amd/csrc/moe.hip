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

#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <array>
#include <mutex>
#include <utility>

#include "qgemm.h"

namespace qm {
namespace {

// ------------------------------------------------------------------ route

constexpr int kRouteThreads = 256;   // one wavefront per token

// (value, index) order used by the router: larger value first, lower index
// on equal values.
__device__ inline void take_better(float& bv, int& be, float ov, int oe) {
  const bool better = ov > bv || (ov == bv && oe < be);
  bv = better ? ov : bv;
  be = better ? oe : be;
}

template <int CTRL>
__device__ inline void dpp_step(float& bv, int& be) {
  const float ov = __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, bv), CTRL, 0xF, 0xF, false));
  const int oe = __builtin_amdgcn_mov_dpp(be, CTRL, 0xF, 0xF, false);
  take_better(bv, be, ov, oe);
}

// Every lane ends with the wavefront's best (value, index): DPP exchanges
// within each row of 16 lanes, then cross-row lane swaps between adjacent
// rows and between the two halves.
__device__ inline void wave_argmax(float& bv, int& be) {
  dpp_step<0xB1>(bv, be);    // quad_perm [1,0,3,2]
  dpp_step<0x4E>(bv, be);    // quad_perm [2,3,0,1]
  dpp_step<0x124>(bv, be);   // row_ror:4
  dpp_step<0x128>(bv, be);   // row_ror:8
  // Every lane now holds its 16-lane row's best.  v_permlane16_swap of a
  // value with itself gives each lane the pair {its row's, the adjacent
  // row's}; v_permlane32_swap the same across the two halves.  The order is
  // symmetric, so the better of each pair is the same in every lane.
  {
    const auto v = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(int, bv), __builtin_bit_cast(int, bv), false, false);
    const auto e = __builtin_amdgcn_permlane16_swap(be, be, false, false);
    bv = __builtin_bit_cast(float, static_cast<int>(v[0]));
    be = static_cast<int>(e[0]);
    take_better(bv, be, __builtin_bit_cast(float, static_cast<int>(v[1])), static_cast<int>(e[1]));
  }
  {
    const auto v = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(int, bv), __builtin_bit_cast(int, bv), false, false);
    const auto e = __builtin_amdgcn_permlane32_swap(be, be, false, false);
    bv = __builtin_bit_cast(float, static_cast<int>(v[0]));
    be = static_cast<int>(e[0]);
    take_better(bv, be, __builtin_bit_cast(float, static_cast<int>(v[1])), static_cast<int>(e[1]));
  }
}

// PER = logits per lane (n_experts <= 64 * PER), a power of two.
template <int PER>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(const float* __restrict__ logits,
                                                              int64_t m, int E, int K,
                                                              int32_t* __restrict__ ids,
                                                              float* __restrict__ gates) {
  const int lane = threadIdx.x & 63;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * (kRouteThreads / 64) + (threadIdx.x >> 6);
  if (t >= m) return;
  const float* row = logits + t * E;
  float v[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = i * 64 + lane;
    v[i] = e < E ? row[e] : -INFINITY;
  }
  uint32_t taken = 0;         // bit i: item i of this lane already selected
  float my_v = -INFINITY;     // lane j < K ends up holding the j-th selected logit
  int my_e = 0;
  for (int j = 0; j < K; ++j) {
    // Lane-local best: highest value, lowest expert index on ties.
    float bv = -INFINITY;
    int be = 0x7FFFFFFF;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = i * 64 + lane;
      const bool ok = e < E && !((taken >> i) & 1u);
      const bool better = ok && (v[i] > bv || (v[i] == bv && e < be));
      bv = better ? v[i] : bv;
      be = better ? e : be;
    }
    // Wavefront argmax with the same order.
    wave_argmax(bv, be);
    if (lane == j) { my_v = bv; my_e = be; }
    if ((be & 63) == lane) taken |= 1u << (be >> 6);
  }
  // Softmax over the selected logits, relative to the largest (slot 0);
  // the denominator is a fixed-order butterfly sum over the lanes.
  const float vmax = __shfl(my_v, 0);
  const float ex = lane < K ? expf(my_v - vmax) : 0.0f;
  float denom = ex;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) denom += __shfl_xor(denom, off);
  if (lane < K) {
    ids[t * K + lane] = my_e;
    gates[t * K + lane] = ex / denom;
  }
}

// ----------------------------------------------------------------- bucket

constexpr int kBucketThreads = 1024;
constexpr int kBucketWaves = kBucketThreads / 64;
constexpr int kBucketUnroll = 8;
// Workgroups: each scatters a contiguous slice of about kBucketSlice
// assignments (two groups of 64 per wavefront), at most kBucketMaxGroups.
constexpr int64_t kBucketSlice = 2048;
constexpr int kBucketMaxGroups = 16;

// Lanes of the wavefront that hold the same expert id (one ballot per bit of
// the id, `bits` = bits needed for n_experts - 1), restricted to the valid
// lanes.
__device__ inline uint64_t match_expert(int e, bool valid, int bits) {
  uint64_t mask = __ballot(valid);
  for (int bit = 0; bit < bits; ++bit) {
    const bool set = (e >> bit) & 1;
    const uint64_t b = __ballot(valid && set);
    mask &= set ? b : ~b;
  }
  return mask;
}

// G workgroups of 16 wavefronts; workgroup g owns the contiguous slice
// [g*S, (g+1)*S) of the assignments and wavefront w of it the contiguous
// part [w*R, (w+1)*R) of that slice.  Pass 1: every workgroup counts all
// assignments per expert, its own per wavefront and the others split into
// those before and after its slice (LDS integer atomics: the counts do not
// depend on the order of the adds).  One pass over the experts then turns
// them into the expert offsets (written by workgroup 0 with the counts) and
// each wavefront's exclusive base: expert offset + assignments of the
// expert before the slice + those of earlier wavefronts in the slice.
// Pass 2 walks the wavefront's part again and places each assignment at
// base + rank among equal experts of its group of 64 lanes, the group's
// leader advancing the base.  The result is the stable counting sort by
// (expert, assignment id), the same for any G.  Groups past the end of a
// range are skipped (wavefront-uniform test).
__global__ __launch_bounds__(kBucketThreads) void bucket_kernel(const int32_t* __restrict__ ids,
                                                                int64_t A, int E,
                                                                int32_t* __restrict__ counts,
                                                                int32_t* __restrict__ offsets,
                                                                int32_t* __restrict__ sorted_assign) {
  __shared__ int base[kBucketWaves][1024];   // per-wavefront counts, then bases
  __shared__ int before[1024], after[1024];  // assignments outside the slice
  __shared__ int wsum[kBucketWaves];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  int bits = 0;
  while ((1 << bits) < E) ++bits;
  for (int w = 0; w < kBucketWaves; ++w) base[w][tid] = 0;
  before[tid] = 0;
  after[tid] = 0;
  __syncthreads();
  const int64_t S = (A + gridDim.x - 1) / gridDim.x;
  const int64_t slo = min<int64_t>(A, blockIdx.x * S), shi = min<int64_t>(A, slo + S);
  const int64_t R = ((shi - slo + kBucketWaves - 1) / kBucketWaves + 63) / 64 * 64;
  const int64_t lo = min<int64_t>(shi, slo + wave * R), hi = min<int64_t>(shi, lo + R);
  const uint64_t lower = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  // kBucketUnroll groups of 64 per round: all their id loads are issued first.
  for (int64_t b0 = lo; b0 < hi; b0 += 64 * kBucketUnroll) {
    int ev[kBucketUnroll];
#pragma unroll
    for (int u = 0; u < kBucketUnroll; ++u) {
      const int64_t a = b0 + u * 64 + lane;
      ev[u] = a < hi ? ids[a] : 0;
    }
#pragma unroll
    for (int u = 0; u < kBucketUnroll; ++u)
      if (b0 + u * 64 + lane < hi) atomicAdd(&base[wave][ev[u]], 1);
  }
  // The assignments outside the slice, strided over all threads.
  auto count_range = [&](int64_t rlo, int64_t rhi, int* dst) {
    for (int64_t b0 = rlo; b0 < rhi; b0 += static_cast<int64_t>(kBucketThreads) * kBucketUnroll) {
      int ev[kBucketUnroll];
#pragma unroll
      for (int u = 0; u < kBucketUnroll; ++u) {
        const int64_t a = b0 + u * kBucketThreads + tid;
        ev[u] = a < rhi ? ids[a] : 0;
      }
#pragma unroll
      for (int u = 0; u < kBucketUnroll; ++u)
        if (b0 + u * kBucketThreads + tid < rhi) atomicAdd(&dst[ev[u]], 1);
    }
  };
  count_range(0, slo, before);
  count_range(shi, A, after);
  __syncthreads();
  // Thread e: total count, per-wavefront exclusive prefix inside the slice;
  // then the exclusive scan of the totals over experts.
  const int e = tid;
  int total = before[e] + after[e];
  for (int w = 0; w < kBucketWaves; ++w) {
    const int c = base[w][e];
    base[w][e] = total - after[e];           // before[e] + earlier wavefronts
    total += c;
  }
  int incl = total;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(incl, d);
    if (lane >= d) incl += o;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int off = incl - total;
  for (int w = 0; w < wave; ++w) off += wsum[w];
  for (int w = 0; w < kBucketWaves; ++w) base[w][e] += off;
  if (blockIdx.x == 0 && e < E) {
    counts[e] = total;
    offsets[e] = off;
  }
  if (blockIdx.x == 0 && e == 0) offsets[E] = static_cast<int32_t>(A);
  __syncthreads();
  for (int64_t b0 = lo; b0 < hi; b0 += 64 * kBucketUnroll) {
    int ev[kBucketUnroll];
#pragma unroll
    for (int u = 0; u < kBucketUnroll; ++u) {
      const int64_t a = b0 + u * 64 + lane;
      ev[u] = a < hi ? ids[a] : 0;
    }
#pragma unroll
    for (int u = 0; u < kBucketUnroll; ++u) {
      if (b0 + u * 64 >= hi) break;                      // wavefront-uniform
      const int64_t a = b0 + u * 64 + lane;
      const bool valid = a < hi;
      const uint64_t mask = match_expert(ev[u], valid, bits);
      const int rank = __popcll(mask & lower);
      if (valid) sorted_assign[base[wave][ev[u]] + rank] = static_cast<int32_t>(a);
      // every lane read its base before the leader advances it (same
      // wavefront, program order); the update is visible to the next group
      if (valid && rank == 0) base[wave][ev[u]] += __popcll(mask);
    }
  }
}

// ---------------------------------------------------------------- combine

// y[t][n] = sum over slots j (in order) of the gate-weighted expert outputs
// (fp16 in the workspace, summed in fp32).  One thread per 8 outputs.
__global__ __launch_bounds__(256) void combine_kernel(const uint16_t* __restrict__ yp, float* __restrict__ y,
                                                      int64_t m, int64_t hidden, int K) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;   // 8-output index
  const int64_t h8 = hidden / 8;
  if (i >= m * h8) return;
  const int64_t t = i / h8, c = i % h8;
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  // Slots in batches of 8: all loads of a batch are in flight before the
  // first add (Yp is read once: nontemporal); the adds keep slot order.
  for (int j0 = 0; j0 < K; j0 += 8) {
    half8v v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (j0 + u < K)
        v[u] = __builtin_nontemporal_load(reinterpret_cast<const half8v*>(yp + (t * K + j0 + u) * hidden) + c);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (j0 + u < K)
#pragma unroll
        for (int r = 0; r < 8; ++r) s[r] += static_cast<float>(v[u][r]);
  }
  float4* dst = reinterpret_cast<float4*>(y + t * hidden) + 2 * c;
  dst[0] = make_float4(s[0], s[1], s[2], s[3]);
  dst[1] = make_float4(s[4], s[5], s[6], s[7]);
}

template <int BMG, int WKG, int BMD, int WKD, int WN, int DG = 2, int DD = 2, bool NT = false, int FMT = QM_Q4_G32>
hipError_t launch_moe_tiles(const MoeArgs& a, hipStream_t st) {
  const int64_t A = a.m * a.top_k;
  // Upper bound on the number of (expert, row tile) pairs: sum of
  // ceil(count_e / BM) <= A / BM + E.  Workgroups past the last tile exit.
  auto tiles = [&](int bm) { return static_cast<unsigned>((A + bm - 1) / bm + a.n_experts); };
  QgemmArgs g{};
  g.counts = a.counts; g.offsets = a.offsets; g.sorted_assign = a.sorted_assign; g.topk_w = a.topk_w;
  g.topk_ids = a.topk_ids;
  g.n_experts = a.n_experts; g.top_k = a.top_k; g.M = A;
  // gate/up + SwiGLU: A = x rows gathered per assignment, N = inter, K = hidden
  g.q = a.gq; g.s = a.gs; g.q2 = a.uq; g.s2 = a.us; g.a = a.x; g.h = a.h; g.N = a.inter; g.K = a.hidden;
  // 1-D grids over (row tile, column block) units, rounded up to whole
  // rounds of XCD chunks (the XCD mapping is done in the kernel).
  auto grid = [&](int bm, int64_t n) {
    const int64_t ny = (padded_rows(n) + 64 * WN - 1) / (64 * WN);
    const int64_t round = static_cast<int64_t>(kXcds) * qg::kMoeChunkTiles * ny;
    const int64_t units = static_cast<int64_t>(tiles(bm)) * ny;
    return dim3(static_cast<unsigned>((units + round - 1) / round * round));
  };
  g.tiles = tiles(BMG);
  hipLaunchKernelGGL((qgemm_kernel<BMG, WN, WKG, QgMode::kMoeGateUp, DG, NT, FMT>), grid(BMG, a.inter), dim3(WN * WKG * 64), 0,
                     st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // down, scaled by the gate weight and scattered to the assignment slot
  g.q = a.dq; g.s = a.ds; g.q2 = nullptr; g.s2 = nullptr; g.a = a.h; g.yp = a.yp; g.N = a.hidden; g.K = a.inter;
  g.tiles = tiles(BMD);
  hipLaunchKernelGGL((qgemm_kernel<BMD, WN, WKD, QgMode::kMoeDown, DD, NT, FMT>), grid(BMD, a.hidden), dim3(WN * WKD * 64), 0,
                     st, g);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n8 = a.m * (a.hidden / 8);
  hipLaunchKernelGGL(combine_kernel, dim3(static_cast<unsigned>((n8 + 255) / 256)), dim3(256), 0, st, a.yp,
                     a.y, a.m, a.hidden, a.top_k);
  return hipGetLastError();
}

}  // namespace

// Scratch of the allocation-free MoE entry point: h and the per-assignment
// outputs of one call, kMoeScratchBytes per device, held by every device the
// library runs on until the process ends.  In host code `scratch` names a
// host-side stand-in, never the device memory: its device address is looked
// up once per device (hipGetSymbolAddress, with that device current) and
// only that address is handed to kernels.  Every call on a device shares the
// same bytes, so calls that overlap on one device race.
static __device__ __align__(256) uint8_t scratch[kMoeScratchBytes];

namespace {
constexpr int kScratchDevices = 64;
void* g_scratch_ptr[kScratchDevices];
hipError_t g_scratch_status[kScratchDevices];
std::once_flag g_scratch_once[kScratchDevices];
}  // namespace

hipError_t moe_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  std::call_once(g_scratch_once[dev], [dev]() {
    void* p = nullptr;
    g_scratch_status[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = g_scratch_status[dev] == hipSuccess ? p : nullptr;
  });
  if (g_scratch_status[dev] != hipSuccess) return g_scratch_status[dev];
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

size_t moe_workspace_bytes(int64_t m, int32_t top_k, int64_t hidden, int64_t inter) {
  const size_t A = static_cast<size_t>(m) * top_k;
  const size_t h_bytes = (A * inter * 2 + 255) / 256 * 256;
  const size_t yp_bytes = (A * hidden * 2 + 255) / 256 * 256;
  return h_bytes + yp_bytes;
}

const char* moe_tile_name(int64_t rows_per_expert) {
  return rows_per_expert <= 24 ? "32-row bucket tiles x 4 panels" : "64-row bucket tiles x 4 panels";
}

hipError_t launch_route(const float* logits, int64_t m, int32_t e, int32_t k, int32_t* ids, float* w,
                        int32_t* counts, int32_t* offsets, int32_t* sorted_assign, hipStream_t st) {
  if (m > 0) {
    const unsigned blocks = static_cast<unsigned>((m + 3) / 4);
    const dim3 g(blocks), b(kRouteThreads);
    if (e <= 64) hipLaunchKernelGGL(route_kernel<1>, g, b, 0, st, logits, m, e, k, ids, w);
    else if (e <= 128) hipLaunchKernelGGL(route_kernel<2>, g, b, 0, st, logits, m, e, k, ids, w);
    else if (e <= 256) hipLaunchKernelGGL(route_kernel<4>, g, b, 0, st, logits, m, e, k, ids, w);
    else if (e <= 512) hipLaunchKernelGGL(route_kernel<8>, g, b, 0, st, logits, m, e, k, ids, w);
    else hipLaunchKernelGGL(route_kernel<16>, g, b, 0, st, logits, m, e, k, ids, w);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  const int64_t A = m * k;
  const unsigned groups = static_cast<unsigned>(
      std::min<int64_t>(kBucketMaxGroups, std::max<int64_t>(1, (A + kBucketSlice - 1) / kBucketSlice)));
  hipLaunchKernelGGL(bucket_kernel, dim3(groups), dim3(kBucketThreads), 0, st, ids, A, e, counts, offsets,
                     sorted_assign);
  return hipGetLastError();
}

hipError_t launch_moe(const MoeArgs& a, int cu_count, hipStream_t st) {
  (void)cu_count;
  // Tuning sweeps only: QM_MOE_PLAN="bm_gate_up,wk_gate_up,bm_down,wk_down,
  // depth_gate_up,depth_down,nontemporal".
  static const std::array<int, 7> forced = [] {
    std::array<int, 7> f{0, 0, 0, 0, 2, 2, 0};
    if (const char* e = tuning_override("QM_MOE_PLAN"))
      std::sscanf(e, "%d,%d,%d,%d,%d,%d,%d", &f[0], &f[1], &f[2], &f[3], &f[4], &f[5], &f[6]);
    return f;
  }();
  using P = std::array<int, 7>;
  if (a.format == QM_Q4_G32) {
    if (forced == P{32, 1, 32, 1, 2, 2, 0}) return launch_moe_tiles<32, 1, 32, 1, 4, 2, 2>(a, st);
    if (forced == P{64, 1, 64, 1, 2, 2, 0}) return launch_moe_tiles<64, 1, 64, 1, 4, 2, 2>(a, st);
    if (forced == P{32, 1, 32, 1, 2, 2, 1}) return launch_moe_tiles<32, 1, 32, 1, 4, 2, 2, true>(a, st);
    if (forced == P{64, 1, 64, 1, 2, 2, 1}) return launch_moe_tiles<64, 1, 64, 1, 4, 2, 2, true>(a, st);
  }
  // Per-chip tile choice by rows per expert: 32-row tiles when buckets are
  // small (decode-like prefill chunks), 64-row tiles otherwise.  While an
  // expert's rows fit one row tile, each weight panel is read by exactly one
  // workgroup: nontemporal weight loads (measured on MI355X with cold caches:
  // 132 -> 102 us at 8 rows per expert, 157 -> 143 us at 32; with several
  // row tiles per expert they lose the L2 reuse between tiles).  Q2 and
  // Q3 use the Q4 plan.  Q5, Q6 and Q8 keep their weights in registers
  // (their LDS stages do not fit beside two workgroups' A stages), and the
  // two-matrix gate/up tile then holds 64 rows only by spilling: their
  // gate/up tiles stay at 32 rows.
  const int64_t rpe = a.m * a.top_k / a.n_experts;
  auto plan = [&](auto f) -> hipError_t {
    constexpr int F = decltype(f)::value;
    if (rpe <= 24) return launch_moe_tiles<32, 1, 32, 1, 4, 2, 2, true, F>(a, st);
    if constexpr (F == QM_Q5_G32 || F == QM_Q6_G32 || F == QM_Q8_G32) {
      return launch_moe_tiles<32, 1, 64, 1, 4, 2, 2, false, F>(a, st);
    } else {
      if (rpe <= 64) return launch_moe_tiles<64, 1, 64, 1, 4, 2, 2, true, F>(a, st);
      return launch_moe_tiles<64, 1, 64, 1, 4, 2, 2, false, F>(a, st);
    }
  };
  switch (a.format) {
    case QM_Q4_G32: return plan(std::integral_constant<int, QM_Q4_G32>{});
    case QM_Q8_G32: return plan(std::integral_constant<int, QM_Q8_G32>{});
    case QM_Q2_G32: return plan(std::integral_constant<int, QM_Q2_G32>{});
    case QM_Q3_G32: return plan(std::integral_constant<int, QM_Q3_G32>{});
    case QM_Q5_G32: return plan(std::integral_constant<int, QM_Q5_G32>{});
    case QM_Q6_G32: return plan(std::integral_constant<int, QM_Q6_G32>{});
    default: return hipErrorInvalidValue;   // F16 / BF16 experts are rejected by the API
  }
}

}  // namespace qm
