// Internal declarations shared by the HIP translation units of libqmatmul.
// Only gfx950 (CDNA4) is targeted: 64-lane wavefronts, fp16 MFMA with fp32
// accumulation, 160 KiB of LDS per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <cstdlib>

#include "../../include/qmatmul.h"

namespace qm {

// Launch-plan overrides for tuning sweeps (QM_GEMV_PLAN, QM_GEMM_PLAN,
// QM_MOE_PLAN) are read only in a library built with -DQM_TUNING_OVERRIDES;
// the shipped library ignores the environment, so a stray variable cannot
// change a production launch.
inline const char* tuning_override(const char* name) {
#ifdef QM_TUNING_OVERRIDES
  return std::getenv(name);
#else
  (void)name;
  return nullptr;
#endif
}

constexpr int kGroup = 32;   // weights per scale (group along K)
constexpr int kPanel = 64;   // rows per device-layout panel (one row per lane)

typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef _Float16 half8v __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));
typedef float float4v __attribute__((ext_vector_type(4)));

__host__ __device__ inline int64_t padded_rows(int64_t n) { return (n + kPanel - 1) / kPanel * kPanel; }

// Workgroups are dealt to the 8 XCDs of an MI355X round-robin by linear
// index, and each XCD has its own L2.  For a grid of `groups` x `per`
// workgroups where the `per` members of a group share cache lines, this maps
// the linear index i to (group, member) so that all members of a group run on
// the same XCD (index i lands on XCD i % 8; members are consecutive among the
// indices of that XCD).  The trailing groups that do not fill all 8 XCDs keep
// the plain mapping.  A bijection on [0, groups * per).
constexpr int kXcds = 8;
__host__ __device__ inline void xcd_group_member(int64_t i, int64_t groups, int per, int64_t* group,
                                                 int* member) {
  const int64_t full = groups / kXcds * kXcds;           // groups in complete sets of 8
  if (i < full * per) {
    const int64_t xcd = i % kXcds, j = i / kXcds;        // j: position among this XCD's indices
    *group = (j / per) * kXcds + xcd;
    *member = static_cast<int>(j % per);
  } else {
    const int64_t r = i - full * per;
    *group = full + r / per;
    *member = static_cast<int>(r % per);
  }
}

// Weight formats: bits per weight, float (no scales) or integer, validity.
__host__ __device__ constexpr int fmt_bits(int32_t fmt) {
  return fmt == QM_Q2_G32 ? 2 : fmt == QM_Q3_G32 ? 3 : fmt == QM_Q4_G32 ? 4 : fmt == QM_Q5_G32 ? 5
       : fmt == QM_Q6_G32 ? 6 : fmt == QM_Q8_G32 ? 8 : 16;
}
__host__ __device__ constexpr bool fmt_float(int32_t fmt) { return fmt == QM_F16 || fmt == QM_BF16; }
__host__ __device__ constexpr bool fmt_valid(int32_t fmt) { return fmt >= QM_Q4_G32 && fmt <= QM_BF16; }
// Bytes of one (panel, group) chunk block of the device layout: 64 rows x 32 codes.
__host__ __device__ constexpr int chunk_block_bytes(int32_t fmt) { return 256 * fmt_bits(fmt); }

// Bytes of codes per row of one matrix (canonical and device layouts agree).
__host__ __device__ inline int64_t row_code_bytes(int32_t fmt, int64_t k) { return k * fmt_bits(fmt) / 8; }
// Scale elements per row (none for the float formats).
__host__ __device__ inline int64_t row_scales(int32_t fmt, int64_t k) { return fmt_float(fmt) ? 0 : k / kGroup; }

// Per-matrix sizes for a layout.
__host__ __device__ inline int64_t matrix_rows(int32_t layout, int64_t n) {
  return layout == QM_LAYOUT_DEVICE ? padded_rows(n) : n;
}

// Error reporting into the thread-local buffer; returns the status.
qm_status fail(qm_status st, const char* fmt, ...);
qm_status check_launch(const char* what);

// Launchers (validated arguments only).
hipError_t launch_quantise(int32_t fmt, const float* w, uint8_t* q, uint16_t* s, int64_t batch,
                           int64_t n, int64_t k, hipStream_t st);
hipError_t launch_dequantise(int32_t fmt, int32_t layout, const uint8_t* q, const uint16_t* s,
                             float* out, int64_t batch, int64_t n, int64_t k, hipStream_t st);
hipError_t launch_repack(int32_t fmt, int32_t src_layout, const uint8_t* sq, const uint16_t* ss,
                         uint8_t* dq, uint16_t* ds, int64_t batch, int64_t n, int64_t k,
                         hipStream_t st);
// Linear workgroup index i (XCD i % 8) -> work unit u, dealing chunks of
// `chunk` consecutive units to the XCDs in turn: the units of one chunk
// (which share operands) run on one XCD, in order, and share its L2, while
// the chunks, and any tail of empty units, spread evenly over the XCDs.  A
// bijection on [0, n) for n a multiple of 8 * chunk.
__host__ __device__ inline int64_t xcd_chunked(int64_t i, int64_t chunk) {
  const int64_t xcd = i % kXcds, j = i / kXcds;
  return ((j / chunk) * kXcds + xcd) * chunk + j % chunk;
}

// Up to kGemmGroupMax matrices with one K sharing A in one grouped GEMM.
constexpr int kGemmGroupMax = 4;

// Up to kGemvGroupMax independent GEMVs with one K and one format.
constexpr int kGemvGroupMax = 8;
struct GemvGroup {
  const uint8_t* q[kGemvGroupMax];
  const uint16_t* s[kGemvGroupMax];
  const uint16_t* x[kGemvGroupMax];
  float* y[kGemvGroupMax];
  int n[kGemvGroupMax];
  int start[kGemvGroupMax + 1];   // first workgroup of each matrix (set by the launcher)
  int count;
  int groups;                     // K / 32
};
// h16 != nullptr: fp16 output into h16 (h unused).
// RMSNorm folded into the GEMVs that consume it: every workgroup forms
// v = x + res (res optional), fp16_RNE(v / rms(v) * w) into LDS as its
// activation, and workgroup 0 writes v to x_out.  Q4 and Q8, K <= 4096.
struct NormArgs {
  const float* x;
  const float* res;
  const uint16_t* w;
  float* x_out;
  float eps;
};
constexpr int64_t kNormGemvMaxK = 4096;
// Largest K whose activation the sub-panel GEMV stages in LDS (16 KiB).
constexpr int kXldsMaxK = 8192;
hipError_t launch_gemv_group_norm(int32_t fmt, GemvGroup& g, const NormArgs& na, int64_t k, int cu_count,
                                  hipStream_t st);
hipError_t launch_gemv_swiglu_norm(int32_t fmt, const uint8_t* qg, const uint16_t* sg, const uint8_t* qu,
                                   const uint16_t* su, const NormArgs& na, float* h, uint16_t* h16, int64_t n,
                                   int64_t k, int cu_count, hipStream_t st);
hipError_t launch_gemv_swiglu(int32_t fmt, const uint8_t* qg, const uint16_t* sg, const uint8_t* qu,
                              const uint16_t* su, const uint16_t* x, float* h, uint16_t* h16, int64_t n, int64_t k,
                              int cu_count, hipStream_t st);
hipError_t launch_gemv_group(int32_t fmt, GemvGroup& g, int64_t k, int cu_count, hipStream_t st);
hipError_t launch_gemv(int32_t fmt, const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y,
                       int64_t n, int64_t k, int cu_count, hipStream_t st);
hipError_t launch_gemm(int32_t fmt, const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y, int64_t m,
                       int64_t n, int64_t k, int cu_count, hipStream_t st);
hipError_t launch_gemm_group(int32_t fmt, int count, const uint8_t* const* q, const uint16_t* const* s,
                             float* const* y, const int64_t* n, const uint16_t* x, int64_t m, int64_t k,
                             int cu_count, hipStream_t st);

// Decode attention: KV rows per workgroup slice and number of slices.
constexpr int kAttnMaxSplits = 256;
constexpr int kAttnScoreFloats = 8192;           // LDS floats for the scores of one slice (32 KiB)
constexpr int64_t kAttnMaxLen = 262144;          // kAttnMaxSplits x (kAttnScoreFloats / 8 heads)
constexpr int64_t kAttnDirectLen = 128;          // caches up to this length: one slice, no merge
struct AttnPlan { int tc; int nsplit; };
AttnPlan attn_decode_plan(int hkv, int group, int64_t len, int cu_count);
size_t attn_decode_workspace_bytes(int32_t hq, int32_t d);
hipError_t launch_attn_decode(const uint16_t* q, const uint16_t* k, const uint16_t* v, int32_t hq, int32_t hkv,
                              int32_t d, int64_t len, int64_t max_len, float scale, float* o, uint16_t* o16,
                              float* ws, int cu_count, hipStream_t st);   // o16 != nullptr: fp16 output

// Causal prefill attention over the cache for a chunk of m query rows
// (workgroups ordered over the device's cu_count CUs; long tiles split over
// key ranges when the workspace holds their partials).  Output: fp32
// [hq][m][d] into o, or, when o16 is set, fp16 rows [m][hq * d] into o16.
struct PrefillPlan {
  int bmax;            // key blocks per split
  int64_t units;       // workgroups of the attention kernel
  int64_t split_tiles; // tiles with more than one split (merge workgroups / heads)
  size_t ws_needed;    // workspace bytes of the unconstrained plan
};
PrefillPlan attn_prefill_plan(int32_t hq, int32_t d, int64_t m, int64_t p0, int cu_count, size_t ws_bytes);
hipError_t launch_attn_prefill(const uint16_t* q, const uint16_t* k, const uint16_t* v, int32_t hq, int32_t hkv,
                               int32_t d, int64_t m, int64_t p0, int64_t max_len, float scale, float* o,
                               uint16_t* o16, void* ws, size_t ws_bytes, int cu_count, hipStream_t st);

// Decode-step glue kernels.
hipError_t launch_embed(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* token, float* x,
                        hipStream_t st);
hipError_t launch_rmsnorm(float* x, const float* res, const uint16_t* w, int64_t rows, int64_t hidden, float eps,
                          uint16_t* out, hipStream_t st);
hipError_t launch_rope_append(const float* q, const float* k, const float* v, int32_t hq, int32_t hkv, int32_t d,
                              int64_t pos, int64_t max_len, float theta, uint16_t* q_out, uint16_t* kc,
                              uint16_t* vc, const uint16_t* q_gain, const uint16_t* k_gain, float eps, const float* table,
                              hipStream_t st);
hipError_t launch_cast_f16(const float* x, int64_t n, uint16_t* y, hipStream_t st);
hipError_t launch_rope_table(int64_t max_len, int32_t d, float theta, float* table, hipStream_t st);
hipError_t launch_rope_table_llama3(int64_t max_len, int32_t d, float theta, float factor, float low, float high,
                                    float orig, float* table, hipStream_t st);
hipError_t launch_embed_rows(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* tokens, int64_t m,
                             float* x, hipStream_t st);
hipError_t launch_rope_append_rows(const float* q, const float* k, const float* v, int32_t hq, int32_t hkv, int32_t d,
                                   int64_t m, int64_t p0, int64_t max_len, float theta, int32_t interleaved,
                                   uint16_t* q_out, uint16_t* kc, uint16_t* vc, const uint16_t* q_gain,
                                   const uint16_t* k_gain, float eps, const float* table, hipStream_t st);
hipError_t launch_heads_to_rows(const float* o, int32_t h, int64_t m, int32_t d, uint16_t* out, hipStream_t st);
hipError_t launch_swiglu(const float* g, const float* u, int64_t n, uint16_t* out, hipStream_t st);

// Epilogue of the fused q/k/v GEMV that applies RoPE and fills the caches:
// W_q and W_k hold each head's rows interleaved (row 2i = row i, row 2i + 1
// = row i + D/2 of the head), so a rotation pair sits in adjacent lanes.
struct QkvRopeEpi {
  uint16_t* q16;        // [Hq][D] rotated queries
  uint16_t* kc;         // [Hkv][max_len][D], row pos written
  uint16_t* vc;
  const float* table;   // [max_len][D/2] (cos, sin)
  int64_t pos;
  int64_t max_len;
  int d;
};
hipError_t launch_gemv_qkv_norm_rope(int32_t fmt, GemvGroup& g, const NormArgs& na, const QkvRopeEpi& epi,
                                     int64_t k, int cu_count, hipStream_t st);
hipError_t launch_argmax(const float* x, int64_t n, int32_t* token, void* ws, hipStream_t st);

struct MoeArgs {
  const uint8_t* gq; const uint16_t* gs;   // gate [E][inter][hidden], device layout
  const uint8_t* uq; const uint16_t* us;   // up   [E][inter][hidden]
  const uint8_t* dq; const uint16_t* ds;   // down [E][hidden][inter]
  const uint16_t* x;                       // [m][hidden] fp16
  const int32_t* counts;                   // [E]
  const int32_t* offsets;                  // [E+1]
  const int32_t* sorted_assign;            // [m*top_k]
  const float* topk_w;                     // [m*top_k]
  const int32_t* topk_ids;                 // [m*top_k]
  float* y;                                // [m][hidden]
  uint16_t* h;                             // workspace: [m*top_k][inter] fp16
  uint16_t* yp;                            // workspace: [m*top_k][hidden] fp16
  int64_t m, hidden, inter;
  int32_t n_experts, top_k;
  int32_t format;                          // of all three expert matrices
};
size_t moe_workspace_bytes(int64_t m, int32_t top_k, int64_t hidden, int64_t inter);
// Bytes of the per-device scratch of qmoe_grouped_gemm_noalloc, and its
// device address on the current device (looked up once per device).
constexpr size_t kMoeScratchBytes = QMOE_NOALLOC_SCRATCH_BYTES;
hipError_t moe_scratch(void** ptr);
hipError_t launch_moe(const MoeArgs& a, int cu_count, hipStream_t st);
hipError_t launch_route(const float* logits, int64_t m, int32_t e, int32_t k, int32_t* ids,
                        float* w, int32_t* counts, int32_t* offsets, int32_t* sorted_assign,
                        hipStream_t st);

// Per-chip choices (Sec. 3.3: per-chip configuration table).
// GEMV launch plan: rows per workgroup (64 = whole panel), wavefronts per
// workgroup, and whether activations are staged in LDS (sub-panel kernel).
// subr: rows per workgroup (64: the panel kernel); waves: wavefronts (panel
// kernel); xlds: x staged in LDS; u: chunks per lane per pass (sub-panel).
struct GemvPlan { int subr; int waves; int xlds; int u; };
GemvPlan gemv_plan(int32_t fmt, int64_t n, int64_t k, int cu_count);
// Name (with template arguments) of the kernel qmatmul_gemv launches for this shape.
void gemv_kernel_name(int32_t fmt, int64_t n, int64_t k, int cu_count, char* buf, size_t len);
struct GemmPlan { int bm; int wn; int wk; };   // rows per tile, panels (wavefronts) per K slice, K slices
GemmPlan gemm_plan(int64_t m, int64_t n, int64_t k, int cu_count);
bool gemm_plan_instantiated(const GemmPlan& p);   // a prefill GEMM tile exists for p
const char* gemm_tile_name(int64_t m, int64_t n);
const char* moe_tile_name(int64_t rows_per_expert);

}  // namespace qm
