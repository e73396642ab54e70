// Decode GEMV with dequantisation fused into the inner loop (BaseRT Sec. 3.3:
// one GEMV kernel per quantisation format for M = 1, weights never
// materialised in dequantised form, traffic cut by the compression ratio).
//
// Mapping on gfx950
//  * one workgroup owns one 64-row panel of the device layout; lane r of
//    every wavefront owns row 64p + r, so one chunk index over the panel is a
//    contiguous 1 KiB (Q4) / 2 KiB (Q8) load: dwordx4 per lane, fully
//    coalesced, no cross-lane reduction inside a wavefront;
//  * the WAVES wavefronts of the workgroup split the K groups of the panel;
//    their per-row partial sums meet once in LDS and wavefront 0 adds them in
//    a fixed order (deterministic, single pass, no workspace, no atomics);
//  * the 32 activations of a group are wavefront-uniform, so they arrive
//    through scalar loads into SGPRs and feed v_dot2_f32_f16 directly;
//  * dequantisation in registers: one v_and_or_b32 turns two offset-binary
//    nibbles u = q + 8 into the fp16 pair 1024 + u (or 1024 + 16u for the
//    nibbles at bits 4-7), one packed fp16 subtraction gives the exact
//    integers q (or 16q), one v_dot2_f32_f16 folds two weights into the
//    fp32 group sum, and the fp16 group scale multiplies the group sum once
//    (about 1.7 VALU operations per Q4 weight).  Q8 builds 0x64|u bytes with
//    v_perm_b32 and subtracts 1152.  Q5/Q6 add their high bit plane into the
//    same fp16 lanes, Q2/Q3 mask crumbs in place with one fp32 sum per bit
//    position, F16 feeds the stored pairs to v_dot2_f32_f16 and BF16 (the
//    upper half of an fp32) goes through fp32 fma with the fp16 activation
//    (Sec. 4.1: eight formats, one kernel each).
#include "qm_internal.h"
#include "rope.h"

#include <hip/hip_fp16.h>

#include <cstdio>
#include <cstdlib>
#include <type_traits>

namespace qm {
namespace {

// fn(std::integral_constant<int, FMT>) for the runtime format (validated by
// the caller).
template <typename Fn>
hipError_t with_format(int32_t fmt, Fn&& fn) {
  switch (fmt) {
    case QM_Q4_G32: return fn(std::integral_constant<int, QM_Q4_G32>{});
    case QM_Q8_G32: return fn(std::integral_constant<int, QM_Q8_G32>{});
    case QM_Q2_G32: return fn(std::integral_constant<int, QM_Q2_G32>{});
    case QM_Q3_G32: return fn(std::integral_constant<int, QM_Q3_G32>{});
    case QM_Q5_G32: return fn(std::integral_constant<int, QM_Q5_G32>{});
    case QM_Q6_G32: return fn(std::integral_constant<int, QM_Q6_G32>{});
    case QM_F16: return fn(std::integral_constant<int, QM_F16>{});
    case QM_BF16: return fn(std::integral_constant<int, QM_BF16>{});
    default: return hipErrorInvalidValue;
  }
}

// Chunks in flight per lane in the panel kernel: 8 Q4 chunks (128 B) or 4
// Q8 chunks (two 16-B halves each), from a per-shape sweep of the lm_head
// sizes on MI355X; about 128 B for the other formats too.
template <int FMT> constexpr int kPanelUnroll = FMT == QM_Q4_G32 ? 8 : FMT == QM_Q8_G32 ? 4
                                              : FMT == QM_Q2_G32 ? 16 : FMT == QM_Q3_G32 ? 8
                                              : FMT == QM_Q5_G32 ? 6 : FMT == QM_Q6_G32 ? 5 : 2;
// Words (dwords) of one lane's chunk: 32 codes of b bits = b dwords.
template <int FMT> constexpr int kWords = fmt_bits(FMT);

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// In the large-matrix kernel weights and scales are streamed once per call:
// nontemporal loads raise the sustained read rate (measured +12% on a plain
// streaming read).  The small-matrix kernel keeps ordinary loads, whose
// first-access latency measured lower.
__device__ __forceinline__ uint4 stream_load16(const uint8_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint32_t stream_load_u16(const uint16_t* p) {
  return __builtin_nontemporal_load(p);
}

// (a & mask) | magic as one v_and_or_b32: the masks live in VGPRs and the
// magic in an SGPR (gfx9 VOP3 takes no literal operand), made opaque once
// per kernel by DequantConsts.
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t mask_v, uint32_t or_s) { return (a & mask_v) | or_s; }

template <int FMT>
struct DequantConsts {
  uint32_t m0, m1, magic;
  uint32_t cm[4], bm[4];      // Q2/Q3: crumb masks 0x00030003 << 2s, Q3 bit masks 0x00040004 << 2s
  __device__ DequantConsts() : m0(0x000F000Fu), m1(0x00F000F0u), magic(0x64006400u) {
    asm volatile("" : "+v"(m0), "+v"(m1));
    asm volatile("" : "+s"(magic));
#pragma unroll
    for (int sc = 0; sc < 4; ++sc) {
      cm[sc] = 0x00030003u << (2 * sc);
      bm[sc] = 0x00040004u << (2 * sc);
      if constexpr (FMT == QM_Q2_G32 || FMT == QM_Q3_G32) asm volatile("" : "+v"(cm[sc]));
      if constexpr (FMT == QM_Q3_G32) asm volatile("" : "+v"(bm[sc]));
    }
  }
};

// Sum over one Q4 group of q[k] * x[k] (fp32).  Dword j of the chunk holds
// the offset-binary nibbles of k = 8j + {0,2,4,6} in bits 0-15 and of
// k = 8j + {1,3,5,7} in bits 16-31, so (dword & 0x000F000F) | 0x6400_6400 is
// the fp16 pair (1024 + u[8j], 1024 + u[8j+1]); the nibbles at bits 4-7 /
// 20-23 land in mantissa bits 4-7 and give (1024 + 16u), i.e. 16*q after
// subtracting 1152.  Those pairs accumulate separately and are scaled by
// 1/16 (exact) at the end of the group.
template <class DC>
__device__ __forceinline__ float dot_q4_chunk(const uint4 w, const uint32_t* xs, const DC& k) {
  const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
  const half2v b1 = {(_Float16)1032.0f, (_Float16)1032.0f};
  const half2v b16 = {(_Float16)1152.0f, (_Float16)1152.0f};
  const uint32_t m0 = k.m0, m1 = k.m1, magic = k.magic;
  float acc1 = 0.0f, acc16 = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t d = wd[j];
    const uint32_t d8 = d >> 8;
    const half2v q01 = __builtin_bit_cast(half2v, and_or(d, m0, magic)) - b1;     // k 0,1
    const half2v q23 = __builtin_bit_cast(half2v, and_or(d, m1, magic)) - b16;    // k 2,3 (x16)
    const half2v q45 = __builtin_bit_cast(half2v, and_or(d8, m0, magic)) - b1;    // k 4,5
    const half2v q67 = __builtin_bit_cast(half2v, and_or(d8, m1, magic)) - b16;   // k 6,7 (x16)
    acc1 = __builtin_amdgcn_fdot2(q01, __builtin_bit_cast(half2v, xs[4 * j + 0]), acc1, false);
    acc16 = __builtin_amdgcn_fdot2(q23, __builtin_bit_cast(half2v, xs[4 * j + 1]), acc16, false);
    acc1 = __builtin_amdgcn_fdot2(q45, __builtin_bit_cast(half2v, xs[4 * j + 2]), acc1, false);
    acc16 = __builtin_amdgcn_fdot2(q67, __builtin_bit_cast(half2v, xs[4 * j + 3]), acc16, false);
  }
  return fmaf(acc16, 0.0625f, acc1);
}

// Sum over 16 Q8 codes (one half chunk, offset-binary bytes) of q * x.
__device__ __forceinline__ float dot_q8_half(const uint4 w, const uint32_t* xs) {
  const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
  const half2v bias = {(_Float16)1152.0f, (_Float16)1152.0f};
  float acc = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t lo = __builtin_amdgcn_perm(0x64646464u, wd[j], 0x04010400u);  // bytes 0,1
    const uint32_t hi = __builtin_amdgcn_perm(0x64646464u, wd[j], 0x04030402u);  // bytes 2,3
    const half2v q0 = __builtin_bit_cast(half2v, lo) - bias;
    const half2v q1 = __builtin_bit_cast(half2v, hi) - bias;
    acc = __builtin_amdgcn_fdot2(q0, __builtin_bit_cast(half2v, xs[2 * j]), acc, false);
    acc = __builtin_amdgcn_fdot2(q1, __builtin_bit_cast(half2v, xs[2 * j + 1]), acc, false);
  }
  return acc;
}

// ---- Activations by lane broadcast (Q4 / Q8 sub-panel rows of 16 or 32).
// Lane l of a 16-lane row holds activation dword l (the fp16 pair
// x[2l], x[2l + 1]) of the group its row of lanes is working on; the dot
// product of pair i takes it from lane i with the DPP row_newbcast:i form of
// v_dot2c_f32_f16, so a chunk needs one 4-byte activation load per lane
// instead of 64 bytes of LDS reads.
//
// The 16 fp16 weight pairs of one chunk, in activation-dword order (pair i
// multiplies dword i).  Q4: (d & 0x000F000F) | 0x6400_6400 is the pair
// (1024 + u) for k even / odd; the nibbles at bits 4-7 give 1024 + 16u, so
// pairs with i % 4 in {1, 3} carry 16q (scaled by 1/16 after the sum).
template <class DC>
__device__ __forceinline__ void q4_pairs(const uint32_t* w, uint32_t* qv, const DC& k) {
  const half2v b1 = {(_Float16)1032.0f, (_Float16)1032.0f};
  const half2v b16 = {(_Float16)1152.0f, (_Float16)1152.0f};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t d = w[j], d8 = d >> 8;
    qv[4 * j + 0] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, and_or(d, k.m0, k.magic)) - b1);
    qv[4 * j + 1] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, and_or(d, k.m1, k.magic)) - b16);
    qv[4 * j + 2] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, and_or(d8, k.m0, k.magic)) - b1);
    qv[4 * j + 3] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, and_or(d8, k.m1, k.magic)) - b16);
  }
}
// Q8: bytes of half h, pairs (0,1), (2,2+1) of dword j -> activation dwords
// 8h + 2j, 8h + 2j + 1.
__device__ __forceinline__ void q8_pairs(const uint32_t* w, uint32_t* qv) {
  const half2v bias = {(_Float16)1152.0f, (_Float16)1152.0f};
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t lo = __builtin_amdgcn_perm(0x64646464u, w[j], 0x04010400u);
    const uint32_t hi = __builtin_amdgcn_perm(0x64646464u, w[j], 0x04030402u);
    qv[2 * j] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, lo) - bias);
    qv[2 * j + 1] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, hi) - bias);
  }
}
// a[i % 4] += dot(pair i of the lane's own qv, activation dword i of its
// row of lanes), i = 0..15.  Hand-written because the compiler does not form
// the DPP variant of v_dot2c itself (it emits a separate v_mov_b32_dpp per
// pair).  The four accumulators put four instructions between writes of one
// register; s_nop 1 before the block covers a VALU write of xd feeding DPP,
// and s_nop 4 after it covers a VALU read of the last results (measured on
// gfx950: with the compiler's single wait state there the final sums were
// read stale).
__device__ __forceinline__ void dpp_dot16(uint32_t xd, const uint32_t* qv, float* a) {
  asm("s_nop 1\n\t"
      "v_dot2c_f32_f16_dpp %0, %4, %5 row_newbcast:0 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %1, %4, %6 row_newbcast:1 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %2, %4, %7 row_newbcast:2 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %3, %4, %8 row_newbcast:3 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %0, %4, %9 row_newbcast:4 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %1, %4, %10 row_newbcast:5 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %2, %4, %11 row_newbcast:6 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %3, %4, %12 row_newbcast:7 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %0, %4, %13 row_newbcast:8 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %1, %4, %14 row_newbcast:9 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %2, %4, %15 row_newbcast:10 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %3, %4, %16 row_newbcast:11 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %0, %4, %17 row_newbcast:12 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %1, %4, %18 row_newbcast:13 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %2, %4, %19 row_newbcast:14 row_mask:0xf bank_mask:0xf\n\t"
      "v_dot2c_f32_f16_dpp %3, %4, %20 row_newbcast:15 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 4"
      : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3])
      : "v"(xd), "v"(qv[0]), "v"(qv[1]), "v"(qv[2]), "v"(qv[3]), "v"(qv[4]), "v"(qv[5]), "v"(qv[6]), "v"(qv[7]),
        "v"(qv[8]), "v"(qv[9]), "v"(qv[10]), "v"(qv[11]), "v"(qv[12]), "v"(qv[13]), "v"(qv[14]), "v"(qv[15]));
}
// One chunk's sum of q * x (before the group scale) with the activations by
// lane broadcast.
template <int FMT, class DC>
__device__ __forceinline__ float dot_chunk_bcast(const uint32_t* w, uint32_t xd, const DC& k) {
  uint32_t qv[16];
  float a[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if constexpr (FMT == QM_Q4_G32) {
    q4_pairs(w, qv, k);
    dpp_dot16(xd, qv, a);
    return fmaf(a[1] + a[3], 0.0625f, a[0] + a[2]);
  } else {
    q8_pairs(w, qv);
    dpp_dot16(xd, qv, a);
    return (a[0] + a[1]) + (a[2] + a[3]);
  }
}

// Sum of v over the lanes l, l ^ 16, l ^ 32, l ^ 48 (from = 16) or l, l ^ 32
// (from = 32), by lane swaps (no LDS); every lane gets the same bits.
template <int FROM>
__device__ __forceinline__ float lane_sum_from(float v) {
  if constexpr (FROM <= 16) {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  }
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

// Shift left by SH (right for negative SH); SH is a constant after unrolling.
__device__ __forceinline__ uint32_t shift_by(uint32_t v, int sh) { return sh >= 0 ? v << sh : v >> -sh; }

// Q5 / Q6: the nibble plane d[0..3] (u & 15, Q4 order) plus u >> 4 from the
// bit plane d[4] (Q5) or the crumb plane d[4..5] (Q6).  As for Q4, the pairs
// from nibble bits 0-3 give 1024 + u and those from bits 4-7 give
// 1024 + 16u; the high part of u is moved to mantissa bit 4 (or 8) of the
// same fp16 lanes with one shift and one v_and_or_b32.  16u <= 1008, so every
// value stays in [1024, 2048), where fp16 is exact on the integers.
template <int FMT>
__device__ __forceinline__ float dot_nib_hi(const uint32_t* d, const uint32_t* xs, const DequantConsts<FMT>& k) {
  constexpr int bias = FMT == QM_Q5_G32 ? 16 : 32;
  const half2v b1 = {(_Float16)(1024 + bias), (_Float16)(1024 + bias)};
  const half2v b16 = {(_Float16)(1024 + 16 * bias), (_Float16)(1024 + 16 * bias)};
  float acc1 = 0.0f, acc16 = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t dj = d[j], dj8 = dj >> 8;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int i = 4 * j + t;                             // pair: codes 2i, 2i+1
      const bool x16 = t & 1;
      const int T = x16 ? 8 : 4;                           // target bit of the high part
      const uint32_t base = and_or(t < 2 ? dj : dj8, x16 ? k.m1 : k.m0, k.magic);
      uint32_t hi;
      if constexpr (FMT == QM_Q5_G32) hi = shift_by(d[4], T - i) & ((1u << T) | (1u << (T + 16)));
      else hi = shift_by(d[4 + i / 8], T - 2 * (i % 8)) & ((3u << T) | (3u << (T + 16)));
      const half2v v = __builtin_bit_cast(half2v, base | hi) - (x16 ? b16 : b1);
      if (x16) acc16 = __builtin_amdgcn_fdot2(v, __builtin_bit_cast(half2v, xs[i]), acc16, false);
      else acc1 = __builtin_amdgcn_fdot2(v, __builtin_bit_cast(half2v, xs[i]), acc1, false);
    }
  }
  return fmaf(acc16, 0.0625f, acc1);
}

// Q2 / Q3: the crumb plane d[0..1] (u & 3) plus, for Q3, u >> 2 from the bit
// plane d[2].  The crumb pair of codes (2i, 2i+1) sits at bits 2t, 16 + 2t
// of its dword (t = i % 8); masking it in place gives 1024 + 4^s u with
// s = t % 4 (the upper four pairs after one shift by 8), the Q3 bit moves to
// bit 2s + 2, and each power 4^s keeps its own fp32 sum, scaled at the end
// (exactly).  4^3 * 7 = 448 keeps every value inside [1024, 2048).
template <int FMT>
__device__ __forceinline__ float dot_crumb(const uint32_t* d, const uint32_t* xs, const DequantConsts<FMT>& k) {
  constexpr int bias = FMT == QM_Q2_G32 ? 2 : 4;
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int cd = 0; cd < 2; ++cd) {
    const uint32_t c = d[cd], c8 = c >> 8;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int i = 8 * cd + t;
      const int sc = t % 4;
      uint32_t v = and_or(t < 4 ? c : c8, k.cm[sc], k.magic);      // masks in VGPRs: one v_and_or_b32
      if constexpr (FMT == QM_Q3_G32) v = and_or(shift_by(d[2], 2 * sc + 2 - i), k.bm[sc], v);
      const _Float16 bb = (_Float16)(1024 + (bias << (2 * sc)));
      const half2v q = __builtin_bit_cast(half2v, v) - half2v{bb, bb};
      acc[sc] = __builtin_amdgcn_fdot2(q, __builtin_bit_cast(half2v, xs[i]), acc[sc], false);
    }
  }
  return acc[0] + acc[1] * 0.25f + acc[2] * 0.0625f + acc[3] * 0.015625f;
}

// F16: fp16 products straight from the stored pairs.  BF16: each bf16 is the
// upper half of an fp32; fp32 fma with the fp16 activation.
__device__ __forceinline__ float dot_f16(const uint32_t* d, const uint32_t* xs) {
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, d[i]), __builtin_bit_cast(half2v, xs[i]), acc, false);
  return acc;
}
__device__ __forceinline__ float dot_bf16(const uint32_t* d, const uint32_t* xs) {
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const half2v xh = __builtin_bit_cast(half2v, xs[i]);
    acc = fmaf(__uint_as_float(d[i] << 16), static_cast<float>(xh[0]), acc);
    acc = fmaf(__uint_as_float(d[i] & 0xFFFF0000u), static_cast<float>(xh[1]), acc);
  }
  return acc;
}

// Sum over one chunk (32 codes of one row and group) of w * x, before the
// group scale (integer formats) or final (float formats).
template <int FMT>
__device__ __forceinline__ float dot_chunk(const uint32_t* d, const uint32_t* xs, const DequantConsts<FMT>& k) {
  if constexpr (FMT == QM_Q4_G32) return dot_q4_chunk(make_uint4(d[0], d[1], d[2], d[3]), xs, k);
  else if constexpr (FMT == QM_Q8_G32)
    return dot_q8_half(make_uint4(d[0], d[1], d[2], d[3]), xs) + dot_q8_half(make_uint4(d[4], d[5], d[6], d[7]), xs + 8);
  else if constexpr (FMT == QM_Q5_G32 || FMT == QM_Q6_G32) return dot_nib_hi<FMT>(d, xs, k);
  else if constexpr (FMT == QM_Q2_G32 || FMT == QM_Q3_G32) return dot_crumb<FMT>(d, xs, k);
  else if constexpr (FMT == QM_F16) return dot_f16(d, xs);
  else return dot_bf16(d, xs);
}

// One lane's share of chunk block `blk` (panel row r): the planes, halves or
// quarters of the device layout, each a coalesced wavefront load.
template <int W, bool NT>
__device__ __forceinline__ void load_words(const uint8_t* p, uint32_t* d) {
  if constexpr (W == 4) {
    const u32x4 v = NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)) : *reinterpret_cast<const u32x4*>(p);
    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
  } else if constexpr (W == 2) {
    const u32x2 v = NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p)) : *reinterpret_cast<const u32x2*>(p);
    d[0] = v.x; d[1] = v.y;
  } else {
    d[0] = NT ? __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p)) : *reinterpret_cast<const uint32_t*>(p);
  }
}
template <int FMT, bool NT>
__device__ __forceinline__ void load_chunk(const uint8_t* blk, int r, uint32_t* d) {
  if constexpr (FMT == QM_Q4_G32) {
    load_words<4, NT>(blk + 16 * r, d);
  } else if constexpr (FMT == QM_Q8_G32) {
    load_words<4, NT>(blk + 16 * r, d);
    load_words<4, NT>(blk + 1024 + 16 * r, d + 4);
  } else if constexpr (FMT == QM_Q2_G32) {
    load_words<2, NT>(blk + 8 * r, d);
  } else if constexpr (FMT == QM_Q3_G32) {
    load_words<2, NT>(blk + 8 * r, d);
    load_words<1, NT>(blk + 512 + 4 * r, d + 2);
  } else if constexpr (FMT == QM_Q5_G32) {
    load_words<4, NT>(blk + 16 * r, d);
    load_words<1, NT>(blk + 1024 + 4 * r, d + 4);
  } else if constexpr (FMT == QM_Q6_G32) {
    load_words<4, NT>(blk + 16 * r, d);
    load_words<2, NT>(blk + 1024 + 8 * r, d + 4);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) load_words<4, NT>(blk + 1024 * j + 16 * r, d + 4 * j);
  }
}

// Group sum -> contribution: times the fp16 group scale (integer formats).
template <int FMT>
__device__ __forceinline__ float scaled_add(uint32_t sbits, float d, float acc) {
  if constexpr (fmt_float(FMT)) return acc + d;
  else return fmaf(__half2float(__ushort_as_half(static_cast<uint16_t>(sbits))), d, acc);
}

// U chunks starting at chunk c (all in range): issue every load, then reduce.
template <int FMT, int U>
__device__ __forceinline__ float gemv_chunks(const uint8_t* __restrict__ q, const uint16_t* __restrict__ s,
                                    const uint32_t* __restrict__ xw, int64_t ch0, int c, int lane,
                                    const DequantConsts<FMT>& k) {
  uint32_t wv[U][kWords<FMT>];
  uint32_t sv[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t ch = ch0 + c + u;
    load_chunk<FMT, true>(q + ch * chunk_block_bytes(FMT), lane, wv[u]);
    if constexpr (!fmt_float(FMT)) sv[u] = stream_load_u16(s + ch * 64 + lane);
    else sv[u] = 0;
  }
  float acc = 0.0f;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint32_t* xs = xw + (c + u) * 16;   // wavefront-uniform: scalar loads
    acc = scaled_add<FMT>(sv[u], dot_chunk<FMT>(wv[u], xs, k), acc);
  }
  return acc;
}

// The last cnt < U chunks of a wavefront's range as one pass: indices past
// the end re-read the last chunk (a valid, cached address) and are not
// reduced, so all loads still go out before the first use.
template <int FMT, int U>
__device__ __forceinline__ float gemv_chunks_tail(const uint8_t* __restrict__ q, const uint16_t* __restrict__ s,
                                         const uint32_t* __restrict__ xw, int64_t ch0, int c, int cnt, int lane,
                                         const DequantConsts<FMT>& k) {
  uint32_t wv[U][kWords<FMT>];
  uint32_t sv[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t ch = ch0 + c + min(u, cnt - 1);
    load_chunk<FMT, true>(q + ch * chunk_block_bytes(FMT), lane, wv[u]);
    if constexpr (!fmt_float(FMT)) sv[u] = stream_load_u16(s + ch * 64 + lane);
    else sv[u] = 0;
  }
  float acc = 0.0f;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (u < cnt) acc = scaled_add<FMT>(sv[u], dot_chunk<FMT>(wv[u], xw + (c + u) * 16, k), acc);   // uniform branch
  }
  return acc;
}

template <int FMT, int WAVES, int U>
__global__ __launch_bounds__(WAVES * 64) void gemv_kernel(const uint8_t* __restrict__ q,
                                                          const uint16_t* __restrict__ s,
                                                          const uint16_t* __restrict__ x,
                                                          float* __restrict__ y, int n_rows,
                                                          int groups, int chunks_per_wave) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t panel = blockIdx.x;
  const int c0 = wave * chunks_per_wave;
  const int c1 = min(groups, c0 + chunks_per_wave);
  const int64_t ch0 = panel * groups;                 // first (panel, group) chunk index
  const uint32_t* xw = reinterpret_cast<const uint32_t*>(x);
  const DequantConsts<FMT> dk;

  float acc = 0.0f;
  int c = c0;
  for (; c + U <= c1; c += U) acc += gemv_chunks<FMT, U>(q, s, xw, ch0, c, lane, dk);
  if constexpr (FMT == QM_Q4_G32 || FMT == QM_Q8_G32) {
    for (; c < c1; ++c) acc += gemv_chunks<FMT, 1>(q, s, xw, ch0, c, lane, dk);
  } else if (c < c1) {
    acc += gemv_chunks_tail<FMT, U>(q, s, xw, ch0, c, c1 - c, lane, dk);
  }

  if (WAVES == 1) {
    const int64_t n = panel * 64 + lane;
    if (n < n_rows) y[n] = acc;
    return;
  }
  __shared__ float part[WAVES][64];
  part[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    float t = part[0][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) t += part[w][lane];
    const int64_t n = panel * 64 + lane;
    if (n < n_rows) y[n] = t;
  }
}

// Sub-panel variant for matrices with fewer 64-row panels than CUs: a
// workgroup owns SUBR rows of one panel (lane = (row r, chunk lane cl), CL =
// 64/SUBR chunk lanes per wavefront), so N/SUBR workgroups spread the VALU
// dequantisation and the loads over many CUs.  One wavefront load reads CL
// contiguous segments of SUBR*16 bytes.  Every lane issues all of its (at
// most kSubU per pass) chunk loads before the first use, so a small GEMV
// costs one memory round trip.  Lanes of a wavefront see different groups,
// so activations come either from an LDS copy of x made once per workgroup
// (XLDS) or straight from global memory (four 16-byte loads per chunk,
// served by the L1/L2 broadcast).  Per-row sums: butterfly over the chunk
// lanes, then a fixed-order sum over wavefronts in LDS.
// Chunks per lane per pass: 8 (F16/BF16: 4, 64 B each).
template <int FMT> constexpr int kSubU = fmt_float(FMT) ? 4 : 8;
// Q4 and Q8 sub-panel workgroups of 16 or 32 rows take their activations by
// lane broadcast (a row of 16 lanes works on one group).
constexpr bool sub_bcast(int fmt, int subr) { return (fmt == QM_Q4_G32 || fmt == QM_Q8_G32) && subr >= 16; }

// One workgroup's share of one matrix: `block` of `nblocks` = N/SUBR.
// SWIGLU: the same rows of a second matrix (q2, s2) go through the same
// loads-then-dots pass, and the workgroup writes silu(a) * b of the two
// row sums a, b (the SwiGLU front half of a feed-forward block).
// The normed activation of a fused RMSNorm, built by every workgroup in LDS
// (xs, fp16, K = 32 * groups <= 4096): v = x + res with 16-byte loads, the
// sum of squares reduced over the workgroup in a fixed order (so every
// workgroup gets the same bits), fp16_RNE(v * inv * w); `write` also stores v
// to x_out.
template <int WAVES>
__device__ __forceinline__ void stage_rmsnorm(const NormArgs& na, int groups, uint4* xs, bool write) {
  constexpr int T = WAVES * 64;
  constexpr int P = (static_cast<int>(kNormGemvMaxK) / 4 + T - 1) / T;   // float4s per thread
  __shared__ float red[WAVES];
  const int n4 = groups * 8;
  const float4* x4 = reinterpret_cast<const float4*>(na.x);
  const float4* r4 = reinterpret_cast<const float4*>(na.res);
  const uint2* w4 = reinterpret_cast<const uint2*>(na.w);
  float4 v[P], r[P];
  uint2 g[P];
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int i = threadIdx.x + j * T;
    const bool ok = i < n4;
    v[j] = ok ? x4[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    g[j] = ok ? w4[i] : make_uint2(0u, 0u);
    r[j] = r4 && ok ? r4[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < P; ++j) {
    v[j].x += r[j].x; v[j].y += r[j].y; v[j].z += r[j].z; v[j].w += r[j].w;
    ss = fmaf(v[j].x, v[j].x, ss);
    ss = fmaf(v[j].y, v[j].y, ss);
    ss = fmaf(v[j].z, v[j].z, ss);
    ss = fmaf(v[j].w, v[j].w, ss);
  }
  if (write) {
    float4* o4 = reinterpret_cast<float4*>(na.x_out);
#pragma unroll
    for (int j = 0; j < P; ++j)
      if (threadIdx.x + j * T < n4) o4[threadIdx.x + j * T] = v[j];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  ss = red[0];
#pragma unroll
  for (int w = 1; w < WAVES; ++w) ss += red[w];
  const float inv = 1.0f / sqrtf(ss / static_cast<float>(groups * 32) + na.eps);
  uint2* xh = reinterpret_cast<uint2*>(xs);
  auto h = [](float f) { const _Float16 t = static_cast<_Float16>(f); return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, t)); };
  auto gf = [](uint32_t b) { return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(b))); };
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int i = threadIdx.x + j * T;
    if (i < n4) {
      const uint32_t a = h(v[j].x * inv * gf(g[j].x & 0xffffu)) | h(v[j].y * inv * gf(g[j].x >> 16)) << 16;
      const uint32_t b = h(v[j].z * inv * gf(g[j].y & 0xffffu)) | h(v[j].w * inv * gf(g[j].y >> 16)) << 16;
      xh[i] = make_uint2(a, b);
    }
  }
}

// Store of the fused q/k/v epilogue: role 0 (q) and 1 (k) rotate the pair
// held by lanes 2i and 2i + 1 (interleaved rows) and write q in fp16 or the
// key into cache row pos; role 2 (v) writes the value row.
__device__ __forceinline__ void qkv_rope_store(const QkvRopeEpi& e, int role, int64_t n, float val, float partner) {
  auto h = [](float f) { const _Float16 t = static_cast<_Float16>(f); return __builtin_bit_cast(uint16_t, t); };
  const int d = e.d, h2 = d / 2;
  const int64_t head = n / d;
  const int w = static_cast<int>(n % d);
  if (role == 2) {
    e.vc[(head * e.max_len + e.pos) * d + w] = h(val);
    return;
  }
  const int i = w >> 1;
  const bool hi = (w & 1) != 0;
  const float2 cs = reinterpret_cast<const float2*>(e.table)[e.pos * h2 + i];
  const float r = hi ? rope_high(partner, val, cs.x, cs.y) : rope_low(val, partner, cs.x, cs.y);
  const int dd = hi ? i + h2 : i;
  if (role == 0)
    e.q16[head * d + dd] = h(r);
  else
    e.kc[(head * e.max_len + e.pos) * d + dd] = h(r);
}

template <int FMT, int SUBR, int WAVES, bool XLDS, bool SWIGLU = false, bool NORM = false, bool QKV_ROPE = false,
          int UP = 0>
__device__ __forceinline__ void gemv_sub_body(const uint8_t* __restrict__ q, const uint16_t* __restrict__ s,
                                              const uint8_t* __restrict__ q2, const uint16_t* __restrict__ s2,
                                              const uint16_t* __restrict__ x, float* __restrict__ y, int n_rows,
                                              int groups, int64_t block, int64_t nblocks,
                                              uint16_t* __restrict__ y16 = nullptr,
                                              const NormArgs* na = nullptr, const QkvRopeEpi* epi = nullptr,
                                              int role = 0) {
  static_assert(!QKV_ROPE || WAVES > 1, "the q/k/v epilogue runs in the multi-wavefront store");
  constexpr int CL = 64 / SUBR;
  constexpr int NM = SWIGLU ? 2 : 1;                  // matrices
  constexpr int U = UP > 0 ? UP : kSubU<FMT>;       // chunks per lane per pass
  extern __shared__ uint4 xs[];                       // groups * 4 uint4 (K halves) if XLDS
  __shared__ float part[NM][WAVES][SUBR];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane % SUBR, cl = lane / SUBR;
  // The CL workgroups of one panel share the 128-byte lines of its scales
  // (and of x): keep them on one XCD so each line is fetched once.
  int64_t panel;
  int sub;
  xcd_group_member(block, nblocks / CL, CL, &panel, &sub);
  const int row = sub * SUBR + r;                     // row inside the panel
  const int64_t ch0 = panel * groups;
  const int stride = WAVES * CL;
  const int first = wave * CL + cl;
  const int iters = (groups + U * stride - 1) / (U * stride);
  const DequantConsts<FMT> dk;
  const uint4* xg = reinterpret_cast<const uint4*>(x);
  // Q4 / Q8 with rows of 16 or 32: activations by lane broadcast, one dword
  // per lane and chunk, from global memory (or from the normed copy in LDS).
  constexpr bool kBcast = sub_bcast(FMT, SUBR);
  const uint32_t* xg32 = reinterpret_cast<const uint32_t*>(x);
  // With x staged in LDS (and no fused norm, no broadcast), one extra
  // wavefront, number WAVES, is the producer of the LDS copy; wavefronts
  // 0 .. WAVES-1 stream the weights.
  constexpr bool kProducer = XLDS && !NORM && !kBcast;

  float acc[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) acc[m] = 0.0f;
  uint32_t wv[U][NM][kWords<FMT>];
  uint32_t sv[U][NM];
  uint32_t xdv[U];                                     // kBcast: the lane's activation dword per chunk
  // Every lane issues all U chunk loads of a pass (chunks past the end of
  // its range re-read the range's last chunk and are discarded by a select):
  // no lane branches between a load and its use, so each dot product waits
  // only for its own chunk's load.
  auto issue = [&](int it) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = min(first + (it * U + u) * stride, groups - 1);
      const int64_t ch = ch0 + c;
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const uint8_t* qm = m == 0 ? q : q2;
        const uint16_t* sm = m == 0 ? s : s2;
        load_chunk<FMT, kBcast>(qm + ch * chunk_block_bytes(FMT), row, wv[u][m]);
        if constexpr (!fmt_float(FMT)) sv[u][m] = sm[ch * 64 + row];
        else sv[u][m] = 0;
      }
      if constexpr (kBcast && !NORM) xdv[u] = xg32[c * 16 + (lane & 15)];
    }
  };
  auto consume = [&](int it) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int craw = first + (it * U + u) * stride;
      const int c = min(craw, groups - 1);
      if constexpr (kBcast) {
        const uint32_t xd = NORM ? reinterpret_cast<const uint32_t*>(xs)[c * 16 + (lane & 15)] : xdv[u];
#pragma unroll
        for (int m = 0; m < NM; ++m) {
          const float t = scaled_add<FMT>(sv[u][m], dot_chunk_bcast<FMT>(wv[u][m], xd, dk), acc[m]);
          acc[m] = craw < groups ? t : acc[m];
        }
      } else {
        uint32_t xv[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint4 t = XLDS ? xs[c * 4 + i] : xg[c * 4 + i];
          xv[4 * i] = t.x; xv[4 * i + 1] = t.y; xv[4 * i + 2] = t.z; xv[4 * i + 3] = t.w;
        }
#pragma unroll
        for (int m = 0; m < NM; ++m) {
          const float t = scaled_add<FMT>(sv[u][m], dot_chunk<FMT>(wv[u][m], xv, dk), acc[m]);
          acc[m] = craw < groups ? t : acc[m];
        }
      }
    }
  };
  if (kProducer && wave == WAVES) {
    // The producer wavefront copies x into LDS (8 loads in flight per lane,
    // clamped indices, duplicates write the same value) and joins the
    // barrier when its writes are complete.
    const int x4 = groups * 4;
    for (int base = 0; base < x4; base += 8 * 64) {
      uint4 t[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) t[j] = xg[min(base + j * 64 + lane, x4 - 1)];
#pragma unroll
      for (int j = 0; j < 8; ++j) xs[min(base + j * 64 + lane, x4 - 1)] = t[j];
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  } else {
    issue(0);
    if constexpr (kProducer) {
      // Wait for x in LDS only: these wavefronts have no LDS writes and their
      // weight loads stay in flight across the (fence-free) barrier.
      asm volatile("s_barrier" ::: "memory");
    } else if constexpr (NORM) {
      stage_rmsnorm<WAVES>(*na, groups, xs, blockIdx.x == 0);
      __syncthreads();
    }
    consume(0);
    for (int it = 1; it < iters; ++it) {
      issue(it);
      consume(it);
    }
  }
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    if constexpr (SUBR >= 16) {
      acc[m] = lane_sum_from<SUBR>(acc[m]);
    } else {
#pragma unroll
      for (int off = SUBR; off < 64; off <<= 1) acc[m] += __shfl_xor(acc[m], off);
    }
  }
  auto out = [&](float a, float b) { return SWIGLU ? a / (1.0f + expf(-a)) * b : a; };
  auto store = [&](int64_t n, float v) {   // y16: fp16 output (round to nearest even) instead of y
    if (y16) {
      const _Float16 hv = static_cast<_Float16>(v);
      y16[n] = __builtin_bit_cast(uint16_t, hv);
    } else {
      y[n] = v;
    }
  };
  if (WAVES == 1) {
    if (lane < SUBR && wave == 0) {              // (wavefront 1, if any, is the producer)
      const int64_t n = panel * 64 + row;
      if (n < n_rows) store(n, out(acc[0], acc[NM - 1]));
    }
    return;
  }
  if (cl == 0 && wave < WAVES) {                 // the producer wavefront has no partial sums
#pragma unroll
    for (int m = 0; m < NM; ++m) part[m][wave][r] = acc[m];
  }
  __syncthreads();
  if (wave == 0 && lane < SUBR) {
    float t[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      t[m] = part[m][0][lane];
#pragma unroll
      for (int w = 1; w < WAVES; ++w) t[m] += part[m][w][lane];
    }
    const int64_t n = panel * 64 + row;
    const float val = out(t[0], t[NM - 1]);
    if constexpr (QKV_ROPE) {
      const float partner = __shfl_xor(val, 1, 64);   // lanes 2i, 2i + 1: one rotation pair (both active)
      if (n < n_rows) qkv_rope_store(*epi, role, n, val, partner);
    } else {
      if (n < n_rows) store(n, val);
    }
  }
}

// Threads of a sub-panel workgroup: WAVES weight-streaming wavefronts, plus
// the producer wavefront of the LDS copy of x when x is staged (no fused norm).
template <int FMT, int SUBR, int WAVES, bool XLDS>
constexpr int kSubThreads = (WAVES + (XLDS && !sub_bcast(FMT, SUBR) ? 1 : 0)) * 64;

template <int FMT, int SUBR, int WAVES, bool XLDS, int U>
__global__ __launch_bounds__((kSubThreads<FMT, SUBR, WAVES, XLDS>)) void gemv_sub_kernel(const uint8_t* __restrict__ q,
                                                              const uint16_t* __restrict__ s,
                                                              const uint16_t* __restrict__ x,
                                                              float* __restrict__ y, int n_rows,
                                                              int groups) {
  // All kernel arguments in one batch of scalar loads (one round trip).
  asm volatile("" ::"s"(q), "s"(s), "s"(x), "s"(y), "s"(n_rows), "s"(groups));
  gemv_sub_body<FMT, SUBR, WAVES, XLDS, false, false, false, U>(q, s, nullptr, nullptr, x, y, n_rows, groups,
                                                                 blockIdx.x, gridDim.x);
}

// SwiGLU pair: h = silu(Wg' x) * (Wu' x) over the same rows, one launch.
template <int FMT, int SUBR, int WAVES, bool XLDS, int U>
__global__ __launch_bounds__((kSubThreads<FMT, SUBR, WAVES, XLDS>)) void gemv_swiglu_kernel(const uint8_t* __restrict__ qg,
                                                                 const uint16_t* __restrict__ sg,
                                                                 const uint8_t* __restrict__ qu,
                                                                 const uint16_t* __restrict__ su,
                                                                 const uint16_t* __restrict__ x,
                                                                 float* __restrict__ h, int n_rows, int groups,
                                                                 uint16_t* __restrict__ h16) {
  asm volatile("" ::"s"(qg), "s"(sg), "s"(qu), "s"(su), "s"(x), "s"(h), "s"(n_rows), "s"(groups), "s"(h16));
  gemv_sub_body<FMT, SUBR, WAVES, XLDS, true, false, false, U>(qg, sg, qu, su, x, h, n_rows, groups, blockIdx.x,
                                                                gridDim.x, h16);
}

// The SwiGLU pair with the RMSNorm of its input folded in.
template <int FMT, int SUBR, int U>
__global__ __launch_bounds__(512) void gemv_swiglu_norm_kernel(const uint8_t* __restrict__ qg,
                                                               const uint16_t* __restrict__ sg,
                                                               const uint8_t* __restrict__ qu,
                                                               const uint16_t* __restrict__ su, NormArgs na,
                                                               float* __restrict__ h, uint16_t* __restrict__ h16,
                                                               int n_rows, int groups) {
  asm volatile("" ::"s"(qg), "s"(sg), "s"(qu), "s"(su), "s"(h), "s"(n_rows), "s"(groups), "s"(h16));
  gemv_sub_body<FMT, SUBR, 8, true, true, true, false, U>(qg, sg, qu, su, nullptr, h, n_rows, groups, blockIdx.x,
                                                          gridDim.x, h16, &na);
}

// A group of independent GEMVs with one K in one launch: the workgroup
// ranges of the matrices follow each other (each but the last rounded up to
// a multiple of 8, so every matrix starts on XCD 0 and keeps the XCD
// grouping of its panels).  Every field of the group is read with
// independent scalar loads and the workgroup's entry is picked by selects,
// so the kernel arguments cost one memory round trip, as for one matrix.
template <int FMT, int SUBR, int WAVES, bool XLDS, int U>
__global__ __launch_bounds__((kSubThreads<FMT, SUBR, WAVES, XLDS>)) void gemv_sub_group_kernel(GemvGroup g) {
  const int b = static_cast<int>(blockIdx.x);
  const uint8_t* q = g.q[0];
  const uint16_t* s = g.s[0];
  const uint16_t* x = g.x[0];
  float* y = g.y[0];
  int n = g.n[0], first = 0;
#pragma unroll
  for (int j = 1; j < kGemvGroupMax; ++j) {
    const bool in = j < g.count && b >= g.start[j];
    q = in ? g.q[j] : q;
    s = in ? g.s[j] : s;
    x = in ? g.x[j] : x;
    y = in ? g.y[j] : y;
    n = in ? g.n[j] : n;
    first = in ? g.start[j] : first;
  }
  int groups = g.groups;
  // Pin every selected field before the branch below, so that the compiler
  // cannot sink their loads past it (one round trip instead of three).
  asm volatile("" ::"s"(q), "s"(s), "s"(x), "s"(y), "s"(n), "s"(first), "s"(groups));
  const int64_t local = b - first;
  const int64_t nb = padded_rows(n) / SUBR;
  if (local >= nb) return;                             // padding workgroup (whole group exits)
  gemv_sub_body<FMT, SUBR, WAVES, XLDS, false, false, false, U>(q, s, nullptr, nullptr, x, y, n, groups, local, nb);
}

// The grouped GEMV with the RMSNorm of the shared input folded in (8
// wavefronts, activation in LDS).
template <int FMT, int SUBR, int U>
__global__ __launch_bounds__(512) void gemv_sub_group_norm_kernel(GemvGroup g, NormArgs na) {
  const int b = static_cast<int>(blockIdx.x);
  const uint8_t* q = g.q[0];
  const uint16_t* s = g.s[0];
  float* y = g.y[0];
  int n = g.n[0], first = 0;
#pragma unroll
  for (int j = 1; j < kGemvGroupMax; ++j) {
    const bool in = j < g.count && b >= g.start[j];
    q = in ? g.q[j] : q;
    s = in ? g.s[j] : s;
    y = in ? g.y[j] : y;
    n = in ? g.n[j] : n;
    first = in ? g.start[j] : first;
  }
  int groups = g.groups;
  asm volatile("" ::"s"(q), "s"(s), "s"(y), "s"(n), "s"(first), "s"(groups));
  const int64_t local = b - first;
  const int64_t nb = padded_rows(n) / SUBR;
  if (local >= nb) return;                             // padding workgroup (never workgroup 0)
  gemv_sub_body<FMT, SUBR, 8, true, false, true, false, U>(q, s, nullptr, nullptr, nullptr, y, n, groups, local, nb,
                                                           nullptr, &na);
}

// The q/k/v projections with the norm folded in and the RoPE / cache
// epilogue (matrix 0: q, 1: k, 2: v).
template <int FMT, int SUBR, int U>
__global__ __launch_bounds__(512) void gemv_qkv_norm_rope_kernel(GemvGroup g, NormArgs na, QkvRopeEpi epi) {
  const int b = static_cast<int>(blockIdx.x);
  const uint8_t* q = g.q[0];
  const uint16_t* s = g.s[0];
  int n = g.n[0], first = 0, role = 0;
#pragma unroll
  for (int j = 1; j < 3; ++j) {
    const bool in = b >= g.start[j];
    q = in ? g.q[j] : q;
    s = in ? g.s[j] : s;
    n = in ? g.n[j] : n;
    first = in ? g.start[j] : first;
    role = in ? j : role;
  }
  int groups = g.groups;
  asm volatile("" ::"s"(q), "s"(s), "s"(n), "s"(first), "s"(groups), "s"(role));
  const int64_t local = b - first;
  const int64_t nb = padded_rows(n) / SUBR;
  if (local >= nb) return;                             // padding workgroup (never workgroup 0)
  gemv_sub_body<FMT, SUBR, 8, true, false, true, true, U>(q, s, nullptr, nullptr, nullptr, nullptr, n, groups, local,
                                                          nb, nullptr, &na, &epi, role);
}

// fn(SUBR, U) with both as integral constants, for the sub-panel plan
// (rows 4 / 8 / 16 / 32; chunks per lane per pass 1, 2, 3, 4 or 8 for Q4 and
// Q8, the format's fixed count otherwise).
template <int FMT, class Fn>
hipError_t with_sub_plan(int subr, int u, Fn&& fn) {
  auto by_u = [&](auto sr) -> hipError_t {
    if constexpr (FMT == QM_Q4_G32 || FMT == QM_Q8_G32) {
      switch (u) {
        case 1: return fn(sr, std::integral_constant<int, 1>{});
        case 2: return fn(sr, std::integral_constant<int, 2>{});
        case 3: return fn(sr, std::integral_constant<int, 3>{});
        case 4: return fn(sr, std::integral_constant<int, 4>{});
        default: return fn(sr, std::integral_constant<int, 8>{});
      }
    } else {
      return fn(sr, std::integral_constant<int, kSubU<FMT>>{});
    }
  };
  switch (subr) {
    case 4: return by_u(std::integral_constant<int, 4>{});
    case 8: return by_u(std::integral_constant<int, 8>{});
    case 16: return by_u(std::integral_constant<int, 16>{});
    default: return by_u(std::integral_constant<int, 32>{});
  }
}

template <int FMT, bool XLDS>
hipError_t launch_sub(const GemvPlan& plan, GemvGroup& g, hipStream_t st) {
  int start = 0;
  for (int i = 0; i < g.count; ++i) {
    g.start[i] = start;
    const int nb = static_cast<int>(padded_rows(g.n[i]) / plan.subr);
    start += i + 1 < g.count ? (nb + kXcds - 1) / kXcds * kXcds : nb;
  }
  g.start[g.count] = start;
  const dim3 grid(static_cast<unsigned>(start));
  const size_t lds = XLDS ? static_cast<size_t>(g.groups) * 64 : 0;
  return with_sub_plan<FMT>(plan.subr, plan.u, [&](auto sr, auto uu) {
    constexpr int SUBR = decltype(sr)::value, U = decltype(uu)::value;
    const dim3 block(kSubThreads<FMT, SUBR, 8, XLDS>);
    if (g.count == 1)
      hipLaunchKernelGGL((gemv_sub_kernel<FMT, SUBR, 8, XLDS, U>), grid, block, lds, st, g.q[0], g.s[0], g.x[0],
                         g.y[0], g.n[0], g.groups);
    else
      hipLaunchKernelGGL((gemv_sub_group_kernel<FMT, SUBR, 8, XLDS, U>), grid, block, lds, st, g);
    return hipGetLastError();
  });
}

template <int FMT>
hipError_t launch_fmt(const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y, int64_t n,
                      int64_t k, int cu_count, hipStream_t st) {
  const int64_t panels = padded_rows(n) / kPanel;
  const int64_t groups = k / kGroup;
  const GemvPlan plan = gemv_plan(FMT, n, k, cu_count);
  if (plan.subr < kPanel) {
    GemvGroup g{};
    g.q[0] = q; g.s[0] = s; g.x[0] = x; g.y[0] = y;
    g.n[0] = static_cast<int>(n); g.count = 1; g.groups = static_cast<int>(groups);
    return plan.xlds ? launch_sub<FMT, true>(plan, g, st) : launch_sub<FMT, false>(plan, g, st);
  }
  const int waves = plan.waves;
  const int cpw = static_cast<int>((groups + waves - 1) / waves);
  const dim3 grid(static_cast<unsigned>(panels));
  const int ni = static_cast<int>(n), gi = static_cast<int>(groups);
  constexpr int U = kPanelUnroll<FMT>;
  switch (waves) {
    case 1: hipLaunchKernelGGL((gemv_kernel<FMT, 1, U>), grid, dim3(64), 0, st, q, s, x, y, ni, gi, cpw); break;
    case 2: hipLaunchKernelGGL((gemv_kernel<FMT, 2, U>), grid, dim3(128), 0, st, q, s, x, y, ni, gi, cpw); break;
    case 4: hipLaunchKernelGGL((gemv_kernel<FMT, 4, U>), grid, dim3(256), 0, st, q, s, x, y, ni, gi, cpw); break;
    default:
      if constexpr (FMT == QM_Q4_G32) {       // only the Q4 plan goes beyond 8 wavefronts
        if (waves == 12) {
          hipLaunchKernelGGL((gemv_kernel<FMT, 12, U>), grid, dim3(768), 0, st, q, s, x, y, ni, gi, cpw);
          break;
        }
        if (waves == 16) {
          hipLaunchKernelGGL((gemv_kernel<FMT, 16, U>), grid, dim3(1024), 0, st, q, s, x, y, ni, gi, cpw);
          break;
        }
      }
      hipLaunchKernelGGL((gemv_kernel<FMT, 8, U>), grid, dim3(512), 0, st, q, s, x, y, ni, gi, cpw);
      break;
  }
  return hipGetLastError();
}

}  // namespace

// Per-chip launch plan, from per-shape sweeps on MI355X (256 CUs).
// Matrices with at least one 64-row panel per CU use the panel kernel.  Q4:
// enough wavefronts per panel for one pass of 8 chunks each (4 at K = 1024,
// 12 at K = 3072), at most 16; other formats: 8 wavefronts (fewer only if
// there are fewer groups).  Smaller matrices use the sub-panel kernel with 8
// wavefronts per workgroup and the smallest row count (8, 16 or 32; from 4
// for N <= 1024 with K >= 2048) that keeps the grid at <= 2 workgroups per
// CU; activations are staged in LDS for K <= 4096 and read from global
// memory beyond.
// Chunks per lane per pass of the sub-panel kernel: enough for one pass over
// the K groups (the smallest of 1, 2, 3, 4, 8 that covers them; 8 and more
// passes beyond), for Q4 and Q8; the format's fixed count otherwise.
static int sub_u(int32_t fmt, int64_t groups, int subr) {
  if (fmt != QM_Q4_G32 && fmt != QM_Q8_G32) return kSubU<QM_Q4_G32> / (fmt_float(fmt) ? 2 : 1);
  const int64_t stride = 8 * (kPanel / subr);
  const int64_t need = (groups + stride - 1) / stride;
  return need <= 1 ? 1 : need <= 2 ? 2 : need <= 3 ? 3 : need <= 4 ? 4 : 8;
}

GemvPlan gemv_plan(int32_t fmt, int64_t n, int64_t k, int cu_count) {
  const int64_t groups = k / kGroup;
  // Tuning sweeps only: QM_GEMV_PLAN="rows,waves,x_in_lds" forces the plan
  // (waves: of the panel kernel, rows = 64; the sub-panel kernel always has 8).
  static const GemvPlan forced = [] {
    GemvPlan f{0, 0, 1, 0};
    if (const char* e = tuning_override("QM_GEMV_PLAN")) std::sscanf(e, "%d,%d,%d", &f.subr, &f.waves, &f.xlds);
    return f;
  }();
  if (forced.subr == 4 || forced.subr == 8 || forced.subr == 16 || forced.subr == 32 || forced.subr == 64) {
    GemvPlan f = forced;
    if (f.subr < kPanel && k > kXldsMaxK) f.xlds = 0;
    if (f.subr == kPanel) {
      int w = 1;
      while (w < 16 && w < f.waves) w = w == 8 ? 12 : (w == 12 ? 16 : 2 * w);
      f.waves = w;
    } else {
      f.waves = 8;
      f.u = sub_u(fmt, groups, f.subr);
      if (sub_bcast(fmt, f.subr)) f.xlds = 0;
    }
    return f;
  }
  const int64_t npad = padded_rows(n);
  const int64_t panels = npad / kPanel;
  GemvPlan p{};
  if (panels >= cu_count) {
    int w = 1;
    if (fmt == QM_Q4_G32) {
      const int64_t want = (groups + kPanelUnroll<QM_Q4_G32> - 1) / kPanelUnroll<QM_Q4_G32>;
      while (w < 16 && w < want) w = w == 8 ? 12 : (w == 12 ? 16 : 2 * w);
    } else {
      while (w < 8 && w * 2 <= groups) w *= 2;
    }
    p.subr = kPanel;
    p.waves = w;
    p.xlds = 0;
    return p;
  }
  int subr = (npad <= 1024 && k >= 2048) ? 4 : 8;
  while (subr < 32 && npad / subr > 2 * cu_count) subr *= 2;
  // Q4 / Q8: at least 16 rows, so the activations go by lane broadcast
  // (measured on MI355X: 16-row workgroups also load faster than 8- or 4-row
  // ones at 3072 -> 3072 and 3072 -> 8192).
  if (fmt == QM_Q4_G32 || fmt == QM_Q8_G32) subr = subr < 16 ? 16 : subr;
  p.subr = subr;
  p.waves = 8;
  p.xlds = sub_bcast(fmt, subr) ? 0 : (k <= kXldsMaxK ? 1 : 0);
  p.u = sub_u(fmt, groups, subr);
  return p;
}

void gemv_kernel_name(int32_t fmt, int64_t n, int64_t k, int cu_count, char* buf, size_t len) {
  const GemvPlan p = gemv_plan(fmt, n, k, cu_count);
  if (p.subr == kPanel)
    std::snprintf(buf, len, "gemv_kernel<%d, %d, %d>", fmt, p.waves,
                  fmt == QM_Q4_G32 ? kPanelUnroll<QM_Q4_G32> : fmt == QM_Q8_G32 ? kPanelUnroll<QM_Q8_G32> : 0);
  else
    std::snprintf(buf, len, "gemv_sub_kernel<%d, %d, %d, %s, %d>", fmt, p.subr, p.waves, p.xlds ? "true" : "false",
                  p.u);
}

hipError_t launch_gemv_group(int32_t fmt, GemvGroup& g, int64_t k, int cu_count, hipStream_t st) {
  int64_t rows = 0;
  for (int i = 0; i < g.count; ++i) rows += padded_rows(g.n[i]);
  if (rows == 0) return hipSuccess;
  const GemvPlan plan = gemv_plan(fmt, rows, k, cu_count);
  if (plan.subr == kPanel) {
    // Enough rows for the panel kernel: one launch per matrix.
    for (int i = 0; i < g.count; ++i) {
      const hipError_t e = launch_gemv(fmt, g.q[i], g.s[i], g.x[i], g.y[i], g.n[i], k, cu_count, st);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  g.groups = static_cast<int>(k / kGroup);
  return with_format(fmt, [&](auto f) {
    constexpr int F = decltype(f)::value;
    return plan.xlds ? launch_sub<F, true>(plan, g, st) : launch_sub<F, false>(plan, g, st);
  });
}

namespace {

template <int FMT>
hipError_t launch_swiglu_fmt(const GemvPlan& plan, const uint8_t* qg, const uint16_t* sg, const uint8_t* qu,
                             const uint16_t* su, const uint16_t* x, float* h, uint16_t* h16, int64_t n, int groups,
                             hipStream_t st) {
  const dim3 grid(static_cast<unsigned>(padded_rows(n) / plan.subr));
  auto go = [&](auto xl) {
    constexpr bool XLDS = decltype(xl)::value;
    const size_t lds = XLDS ? static_cast<size_t>(groups) * 64 : 0;
    return with_sub_plan<FMT>(plan.subr, plan.u, [&](auto sr, auto uu) {
      constexpr int SUBR = decltype(sr)::value, U = decltype(uu)::value;
      hipLaunchKernelGGL((gemv_swiglu_kernel<FMT, SUBR, 8, XLDS, U>), grid, dim3(kSubThreads<FMT, SUBR, 8, XLDS>), lds, st, qg,
                         sg, qu, su, x, h, static_cast<int>(n), groups, h16);
      return hipGetLastError();
    });
  };
  return plan.xlds ? go(std::true_type{}) : go(std::false_type{});
}

}  // namespace

// The sub-panel plan of one matrix of N rows (each workgroup covers its rows
// of both matrices); matrices large enough for the panel kernel use 32-row
// workgroups, 8 wavefronts.
hipError_t launch_gemv_swiglu(int32_t fmt, const uint8_t* qg, const uint16_t* sg, const uint8_t* qu,
                              const uint16_t* su, const uint16_t* x, float* h, uint16_t* h16, int64_t n, int64_t k,
                              int cu_count, hipStream_t st) {
  if (n == 0) return hipSuccess;
  GemvPlan plan = gemv_plan(fmt, n, k, cu_count);
  if (plan.subr == kPanel) {
    plan.subr = 32;
    plan.xlds = sub_bcast(fmt, 32) ? 0 : (k <= kXldsMaxK ? 1 : 0);
    plan.u = sub_u(fmt, k / kGroup, 32);
  }
  const int groups = static_cast<int>(k / kGroup);
  return with_format(fmt, [&](auto f) {
    return launch_swiglu_fmt<decltype(f)::value>(plan, qg, sg, qu, su, x, h, h16, n, groups, st);
  });
}

// Fused RMSNorm + GEMVs: the sub-panel plan of the rows (32-row workgroups
// where the plan would take the panel kernel), always 8 wavefronts with the
// activation in LDS.
static int norm_subr(int32_t fmt, int64_t rows, int64_t k, int cu_count) {
  const GemvPlan plan = gemv_plan(fmt, rows, k, cu_count);
  return plan.subr == kPanel ? 32 : plan.subr;
}

hipError_t launch_gemv_qkv_norm_rope(int32_t fmt, GemvGroup& g, const NormArgs& na, const QkvRopeEpi& epi,
                                     int64_t k, int cu_count, hipStream_t st) {
  int64_t rows = 0;
  for (int i = 0; i < 3; ++i) rows += padded_rows(g.n[i]);
  const int subr = norm_subr(fmt, rows, k, cu_count);
  g.groups = static_cast<int>(k / kGroup);
  int start = 0;
  for (int i = 0; i < 3; ++i) {
    g.start[i] = start;
    const int nb = static_cast<int>(padded_rows(g.n[i]) / subr);
    start += i + 1 < 3 ? (nb + kXcds - 1) / kXcds * kXcds : nb;
  }
  g.start[3] = start;
  const dim3 grid(static_cast<unsigned>(start));
  const size_t lds = static_cast<size_t>(g.groups) * 64;
  const int u = sub_u(fmt, g.groups, subr);
  auto go = [&](auto f) -> hipError_t {
    constexpr int F = decltype(f)::value;
    return with_sub_plan<F>(subr, u, [&](auto sr, auto uu) {
      hipLaunchKernelGGL((gemv_qkv_norm_rope_kernel<F, decltype(sr)::value, decltype(uu)::value>), grid, dim3(512),
                         lds, st, g, na, epi);
      return hipGetLastError();
    });
  };

  return with_format(fmt, go);
}

hipError_t launch_gemv_group_norm(int32_t fmt, GemvGroup& g, const NormArgs& na, int64_t k, int cu_count,
                                  hipStream_t st) {
  int64_t rows = 0;
  for (int i = 0; i < g.count; ++i) rows += padded_rows(g.n[i]);
  const int subr = norm_subr(fmt, rows, k, cu_count);
  g.groups = static_cast<int>(k / kGroup);
  int start = 0;
  for (int i = 0; i < g.count; ++i) {
    g.start[i] = start;
    const int nb = static_cast<int>(padded_rows(g.n[i]) / subr);
    start += i + 1 < g.count ? (nb + kXcds - 1) / kXcds * kXcds : nb;
  }
  g.start[g.count] = start;
  const dim3 grid(static_cast<unsigned>(start));
  const size_t lds = static_cast<size_t>(g.groups) * 64;
  const int u = sub_u(fmt, g.groups, subr);
  auto go = [&](auto f) -> hipError_t {
    constexpr int F = decltype(f)::value;
    return with_sub_plan<F>(subr, u, [&](auto sr, auto uu) {
      hipLaunchKernelGGL((gemv_sub_group_norm_kernel<F, decltype(sr)::value, decltype(uu)::value>), grid, dim3(512),
                         lds, st, g, na);
      return hipGetLastError();
    });
  };

  return with_format(fmt, go);
}

hipError_t launch_gemv_swiglu_norm(int32_t fmt, const uint8_t* qg, const uint16_t* sg, const uint8_t* qu,
                                   const uint16_t* su, const NormArgs& na, float* h, uint16_t* h16, int64_t n,
                                   int64_t k, int cu_count, hipStream_t st) {
  const int subr = norm_subr(fmt, n, k, cu_count);
  const int groups = static_cast<int>(k / kGroup);
  const dim3 grid(static_cast<unsigned>(padded_rows(n) / subr));
  const size_t lds = static_cast<size_t>(groups) * 64;
  const int ni = static_cast<int>(n);
  const int u = sub_u(fmt, groups, subr);
  auto go = [&](auto f) -> hipError_t {
    constexpr int F = decltype(f)::value;
    return with_sub_plan<F>(subr, u, [&](auto sr, auto uu) {
      hipLaunchKernelGGL((gemv_swiglu_norm_kernel<F, decltype(sr)::value, decltype(uu)::value>), grid, dim3(512),
                         lds, st, qg, sg, qu, su, na, h, h16, ni, groups);
      return hipGetLastError();
    });
  };

  return with_format(fmt, go);
}

hipError_t launch_gemv(int32_t fmt, const uint8_t* q, const uint16_t* s, const uint16_t* x, float* y,
                       int64_t n, int64_t k, int cu_count, hipStream_t st) {
  if (n == 0) return hipSuccess;
  return with_format(fmt, [&](auto f) { return launch_fmt<decltype(f)::value>(q, s, x, y, n, k, cu_count, st); });
}

}  // namespace qm
