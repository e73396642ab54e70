/*
 * qmatmul.h -- C ABI of the MI355X (gfx950) weight-only-quantised matmul library.
 *
 * The library implements the matrix products of LLM decode and prefill with
 * quantised weights: a fused dequantise+GEMV for batch-1 decode, a
 * dequantise-into-LDS + fp16 MFMA GEMM for prefill, and the top-k-routed
 * grouped expert GEMM of a mixture-of-experts layer; plus grouped-query
 * attention over a pre-allocated KV cache for decode and causal
 * FlashAttention for prefill chunks; plus the rest of a dense decode step
 * (embedding, RMSNorm, RoPE with the cache append, greedy sampling), folded
 * into the matmuls where that removes a launch (BaseRT, Sec. 3.3
 * "Kernel Fusion and Specialisation": one GEMV (M = 1) and one GEMM (M > 1)
 * kernel per quantisation format, dequantisation inside the inner loop and
 * never materialised; Sec. 3.4 "Prefill": tiled GEMM for prompts, bounded
 * chunks, FlashAttention; Sec. 3.2: the KV cache; Sec. 4.1: the weight
 * formats and the MoE models).
 *
 * Conventions shared by every entry point
 *  - Pointers named d_* / device buffers are HIP device pointers; the caller
 *    owns every buffer, workspaces included.  The library never allocates,
 *    frees or retains memory (Sec. 3.2, "Zero-Allocation Decode Loop").
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    QM_OK means "validated and enqueued on stream"; nothing is synchronised.
 *  - Arguments are validated on the host before anything is enqueued.  On an
 *    error nothing is enqueued, outputs are untouched and a message is left in
 *    a thread-local buffer read by qm_last_error() (Sec. 3.2: the error path
 *    uses a fixed per-thread buffer too).
 *  - A launch failure reported by the HIP runtime maps to QM_EDEVICE.
 *  - Calls that share output or workspace buffers and overlap on one device
 *    race; the library holds no state besides an immutable per-device
 *    configuration table.
 *
 * Weight formats (Sec. 4.1: Q2, Q3, Q4, Q5, Q6, Q8, BF16 and FP16)
 *  Integer formats Qb (b = 2, 3, 4, 5, 6, 8 bits), group-32 symmetric, one
 *  fp16 scale per 32 weights along K.  For row n and group g = k / 32 of a
 *  weight matrix W [N][K]:
 *    m = max |w| over the group (fp32), s32 = m / qmax (fp32, correctly
 *    rounded), s16 = fp16_RNE(s32), s = value(s16);
 *    q = 0 if s == 0, else clamp(rint_half_even(w / s), lo, hi)  (fp32 division);
 *    qmax = 2^(b-1) - 1 and [lo, hi] = [-2^(b-1), 2^(b-1) - 1], except Q8:
 *    qmax = 127, [lo, hi] = [-127, 127].  (Q2: qmax 1, Q3: 3, Q4: 7, Q5: 15,
 *    Q6: 31.)  The dequantised weight is w' = s * q, exact in fp32.
 *  Float formats F16 and BF16: w is rounded to fp16 / bf16 (round to nearest
 *  even; fp16 subnormals kept) and w' is that value; there are no scales
 *  (the scale buffer has 0 bytes and `scales` may be NULL).
 *
 *  CANONICAL layout (QM_LAYOUT_CANONICAL):
 *    Qb codes: per row a little-endian bit stream of K*b/8 bytes; code k is
 *              the b-bit two's complement of q at bits b*k .. b*k + b - 1
 *              (bit i of the stream is bit i%8 of byte i/8).  So Q4 byte j =
 *              (q[2j] & 0xF) | ((q[2j+1] & 0xF) << 4) and Q8 is int8 [N][K];
 *    F16/BF16: uint16 [N][K] bit patterns;
 *    scales:   uint16 [N][K/32], fp16 bit patterns.
 *
 *  DEVICE layout (QM_LAYOUT_DEVICE), the one the matmul kernels read: rows
 *  are grouped into panels of 64 (N is padded up to a multiple of 64 with
 *  zero bytes), and the 32 codes of one (row, group) form a "chunk"; the
 *  chunks of one (panel p = n/64, group g) lie together at byte
 *  (p*G + g) * CB, G = K/32, r = n%64, CB the chunk block size below.
 *  Integer codes are stored offset-binary, u = q + 2^(b-1) (Q8: q + 128).
 *    Q4 (CB 1024): row r's 16 bytes at 16r.  Dword j covers k = 8j .. 8j+7
 *        of the group; its nibble t (bits 4t..4t+3) holds u of k-offset 2t
 *        (t < 4) or 2(t-4)+1 (t >= 4).
 *    Q8 (CB 2048): two 16-byte halves h = 0, 1 (k = 16h .. 16h+15); half h of
 *        row r at h*1024 + 16r, byte i = u of k = 16h + i.
 *    Q2, Q3, Q5, Q6: u is split into bit planes, each plane 64 rows of equal
 *        size, one after the other:
 *          nibble plane (16 B a row, u & 15), order as Q4;
 *          crumb plane (8 B a row): dword j, bits 2t..2t+1 hold k = 16j + 2t
 *            and bits 16+2t..17+2t hold k = 16j + 2t + 1 (t = 0..7);
 *          bit plane (4 B a row): bit t holds k = 2t, bit 16+t holds k = 2t+1.
 *        Q2 (CB 512):  crumbs of u.
 *        Q3 (CB 768):  crumbs of u & 3 (512 B), then bits of u >> 2 (256 B).
 *        Q5 (CB 1280): nibbles of u & 15 (1024 B), then bits of u >> 4.
 *        Q6 (CB 1536): nibbles of u & 15 (1024 B), then crumbs of u >> 4.
 *    F16/BF16 (CB 4096): four 16-byte quarters j = 0..3 (k = 8j .. 8j+7, in
 *        order); quarter j of row r at j*1024 + 16r.
 *    scales: uint16 at element (p*G + g)*64 + r.
 *  Stacked matrices (batch > 1, e.g. the experts of a MoE layer) place
 *  matrix b at b * (bytes of one matrix) in both buffers, in both layouts.
 *  Every 64-lane wavefront load of one plane (or half, or quarter) of a chunk
 *  block reads contiguous bytes, so the weight stream is fully coalesced.
 */
#ifndef QMATMUL_H
#define QMATMUL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  QM_OK = 0,
  QM_EINVAL = 1,      /* null pointer, bad enum, negative size            */
  QM_ESHAPE = 2,      /* K % 32 != 0, mismatched shapes, size limits      */
  QM_EALIGN = 3,      /* a device pointer is not 16-byte aligned          */
  QM_EFORMAT = 4,     /* unsupported format for this entry point          */
  QM_ELAYOUT = 5,     /* wrong layout for this entry point                */
  QM_EWORKSPACE = 6,  /* workspace missing or smaller than required       */
  QM_EDEVICE = 7      /* the HIP runtime reported an error                */
} qm_status;

enum {
  QM_Q4_G32 = 1, QM_Q8_G32 = 2, QM_Q2_G32 = 3, QM_Q3_G32 = 4, QM_Q5_G32 = 5, QM_Q6_G32 = 6,
  QM_F16 = 7, QM_BF16 = 8
};
enum { QM_LAYOUT_CANONICAL = 0, QM_LAYOUT_DEVICE = 1 };

/* Non-owning view of a quantised weight tensor [batch][n][k].
 * qdata: device codes in `layout`; scales: device fp16 bits (unused, may be
 * NULL, for F16/BF16).  k % 32 == 0.  Both pointers must be 16-byte aligned;
 * the buffers must hold at least the sizes qm_weight_bytes() returns for
 * (format, layout, batch, n, k). */
typedef struct {
  int32_t format;
  int32_t layout;
  int64_t batch;
  int64_t n;
  int64_t k;
  void* qdata;
  uint16_t* scales;
} qm_qweight;

/* Text of the last error on the calling thread ("" if none yet), kept in a
 * fixed per-thread buffer (Sec. 3.2: reporting an error allocates nothing
 * either).  The pointer stays valid until the next failing call on the same
 * thread. */
const char* qm_last_error(void);

/* Host-only: bytes of the code buffer and of the scale buffer for a tensor
 * [batch][n][k] in the given format and layout (DEVICE pads n to 64), so the
 * caller can allocate every buffer up front (Sec. 3.2: nothing is allocated
 * on the hot path; Sec. 4.1: the weight formats). */
qm_status qm_weight_bytes(int32_t format, int32_t layout, int64_t batch, int64_t n,
                          int64_t k, size_t* qbytes, size_t* sbytes);

/* Offline conversion of fp32 weights into one of the quantised formats the
 * runtime executes (Sec. 4.1: Q2 ... Q8, BF16 and FP16 weights; Sec. 3.3:
 * weights stay quantised and are dequantised inside the matmul kernels).
 * Quantise fp32 weights w [batch][n][k] (device, row-major) into `out`, which
 * must be in CANONICAL layout with out->format set.  Bit-exact with the
 * format definition above (one thread per group, IEEE fp32 division,
 * round-half-even, fp16 round-to-nearest-even; F16/BF16: one rounding per
 * weight).  Weights must be finite and every group's max|w| / qmax must be
 * <= 65504 (F16: every |w| below 65520), not scanned. */
qm_status qm_quantise(int32_t format, const float* w, const qm_qweight* out, void* stream);

/* Dequantise w (either layout) into fp32 out [batch][n][k] (device):
 * out = s * q, exact.  Not on the hot path, where dequantisation happens in
 * the matmul's inner loop and is never materialised (Sec. 3.3); this is the
 * reference view of the weights the kernels compute with. */
qm_status qm_dequantise(const qm_qweight* w, float* out, void* stream);

/* Reorder codes and scales between layouts (CANONICAL <-> DEVICE), the
 * device layout being chosen for coalesced access (Sec. 3.2: memory layouts
 * chosen to maximise coalesced access; Sec. 1.1: memory-aware data layout).
 * src and dst must agree in format, batch, n, k and differ in layout; the map is a
 * bijection on the real rows, and DEVICE padding rows are written as zero.
 * src and dst buffers must not overlap. */
qm_status qm_repack(const qm_qweight* src, const qm_qweight* dst, void* stream);

/* Decode GEMV (Sec. 3.3, M = 1): y[n] = sum_k w'[n][k] * x[k].
 * w: DEVICE layout, batch 1, any format (one kernel per format).  x: fp16
 * [k] (device).  y: fp32 [n] (device).  Dequantisation happens in
 * registers; products and sums in fp32.
 * Single kernel launch, no workspace, deterministic. */
qm_status qmatmul_gemv(const qm_qweight* w, const uint16_t* x, float* y, void* stream);

/* SwiGLU front half of a feed-forward block at batch 1 (Sec. 3.3: the
 * activation fused into the producing kernel, saving a launch and a
 * global-memory round trip):
 *   h[n] = silu(g[n]) * u[n],  g = Wg' x,  u = Wu' x,  silu(z) = z / (1 + e^-z).
 * w_gate, w_up: DEVICE layout, batch 1, the same format (any) and the
 * same n and k.  x: fp16 [k] (16-byte aligned); h: fp32 [n].  g and u are
 * accumulated as in qmatmul_gemv (fp32), in one pass over the same rows of
 * both matrices.  Deterministic. */
qm_status qmatmul_gemv_swiglu(const qm_qweight* w_gate, const qm_qweight* w_up, const uint16_t* x, float* h,
                              void* stream);

/* As qmatmul_gemv_swiglu, with h written as fp16 [n] (round to nearest
 * even of the same fp32 value; 2-byte aligned), ready to be the input of
 * the down projection's GEMV.
 * (Sec. 3.3: the fp16 conversion fused into the producer.) */
qm_status qmatmul_gemv_swiglu_f16(const qm_qweight* w_gate, const qm_qweight* w_up, const uint16_t* x, uint16_t* h,
                                  void* stream);

/* RMSNorm folded into the GEMVs that read its output (Sec. 3.3: each fusion
 * removes a launch; Sec. 3.2: normalisation kernels).  With
 *   v = x + residual (residual may be NULL: v = x),
 *   n = fp16_RNE(v / sqrt(mean(v^2) + eps) * gain):
 * qmatmul_gemv_grouped_rmsnorm: y_i = w_i' n for i < count (the q/k/v
 * projections of a layer), as qmatmul_gemv_grouped with every x_i = n;
 * qmatmul_gemv_swiglu_rmsnorm_f16: h = fp16_RNE(silu(Wg' n) * (Wu' n)), as
 * qmatmul_gemv_swiglu_f16.  Both write v to x_out (fp32 [k]), the residual
 * stream for the next fused call, which must not overlap x or residual.
 * x, residual, x_out: fp32 [k], 16-byte aligned; gain: fp16 [k], 8-byte
 * aligned.  Weights: any of the eight formats (one per call), DEVICE layout, batch 1, one k <= 4096, every
 * n >= 1.  Every workgroup recomputes n into LDS from x and residual (the
 * sum of squares in fp32, in the same order in every workgroup); workgroup 0
 * writes x_out.  One launch each. */
qm_status qmatmul_gemv_grouped_rmsnorm(int32_t count, const qm_qweight* w, const float* x, const float* residual,
                                       const uint16_t* gain, float eps, float* x_out, float* const* y, void* stream);
qm_status qmatmul_gemv_swiglu_rmsnorm_f16(const qm_qweight* w_gate, const qm_qweight* w_up, const float* x,
                                          const float* residual, const uint16_t* gain, float eps, float* x_out,
                                          uint16_t* h, void* stream);

/* ---- Glue of a prompt (prefill) chunk of m tokens (Sec. 3.4: chunked
 * prefill; the same operations as a decode step over m rows, with the GEMMs
 * and qattn_prefill between them). */

/* x[r] = table[tokens[r]] (fp16 -> fp32), r < m; x: fp32 [m][hidden];
 * tokens: int32 [m] on the device; ids outside [0, vocab) give NaN rows.
 * 0 <= m <= 32768.
 * (Sec. 3.4: chunked prefill; Sec. 3.2: embedding kernel.) */
qm_status qdec_embed_rows(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* tokens, int64_t m,
                          float* x, void* stream);

/* RoPE and the cache append for tokens r < m at positions p0 + r:
 * q: fp32 [m][n_q_heads * head_dim], k, v: fp32 [m][n_kv_heads * head_dim]
 * (GEMM outputs; with interleaved = 1 each head's dimensions of q and k are
 * in the interleaved order of qmatmul_gemv_qkv_rmsnorm_rope's weights);
 * q_out: fp16 [n_q_heads][m][head_dim] (qattn_prefill's layout), rotated;
 * cache rows p0 .. p0 + m - 1 written (keys rotated).  Rotation as
 * qdec_rope_append, the per-head norms too.  head_dim 64 or 128;
 * 1 <= m <= 32768; p0 + m <= max_len <= 262144; theta > 1.
 * table: NULL, or qdec_rope_table's (cos, sin) pairs for this head_dim and
 * theta over table_len >= p0 + m positions (8-byte aligned), read instead
 * of computing each angle (the same values; the kernel then skips the fp64
 * angle, cosine and sine per element).  A table of another theta gives
 * other rotations, not an error.
 * (Sec. 3.4: chunked prefill; Sec. 3.2: RoPE and the KV cache.) */
qm_status qdec_rope_append_rows(const float* q, const float* k, const float* v, int32_t n_q_heads,
                                int32_t n_kv_heads, int32_t head_dim, int64_t m, int64_t p0, int64_t max_len,
                                float theta, int32_t interleaved, const uint16_t* q_norm, const uint16_t* k_norm,
                                float eps, const float* table, int64_t table_len, uint16_t* q_out,
                                uint16_t* k_cache, uint16_t* v_cache, void* stream);

/* out[r][h * head_dim + d] = fp16_RNE(o[h][r][d]): qattn_prefill's output
 * as the output projection's GEMM input.
 * (Sec. 3.4: chunked prefill, the attention output handed to the next GEMM.) */
qm_status qdec_heads_to_rows_f16(const float* o, int32_t n_heads, int64_t m, int32_t head_dim, uint16_t* out,
                                 void* stream);

/* out[i] = fp16_RNE(silu(gate[i]) * up[i]), i < n (fp32 in): the SwiGLU of
 * the prompt's gate/up GEMM outputs.
 * (Sec. 3.4: chunked prefill; Sec. 3.2: activation kernels.) */
qm_status qdec_swiglu_f16(const float* gate, const float* up, int64_t n, uint16_t* out, void* stream);

/* (cos, sin) table of the rotary embedding for every position of a cache:
 * table[p][i] = (cos a, sin a), a = p * theta^(-2i/head_dim), i < head_dim/2,
 * p < max_len, angle in fp64, fp32 entries (the values qdec_rope_append
 * computes).  table: fp32 [max_len][head_dim/2][2], 8-byte aligned.  Built
 * once per cache (Sec. 3.2: RoPE). */
qm_status qdec_rope_table(int64_t max_len, int32_t head_dim, float theta, float* table, void* stream);

/* The same table for the Llama 3 models' long-context RoPE (the Llama 3.2
 * models of Sec. 4 carry it; the paper does not restate it): each pair's
 * frequency f = theta^(-2i/head_dim), of wavelength w = 2 pi / f, is kept
 * while w < original_len / high_freq_factor, divided by factor while
 * w > original_len / low_freq_factor, and in between blended as
 * (1 - t) f / factor + t f, t = (original_len / w - low_freq_factor) /
 * (high_freq_factor - low_freq_factor); a = p * f in fp64.  Needs finite
 * factor >= 1, 0 < low_freq_factor < high_freq_factor, original_len > 0
 * (else QM_EINVAL); shapes, alignment and layout as qdec_rope_table.  Every
 * entry point that takes a (cos, sin) table applies it as given, so a decoder
 * that passes this table everywhere runs the scaled RoPE. */
qm_status qdec_rope_table_llama3(int64_t max_len, int32_t head_dim, float theta, float factor, float low_freq_factor,
                                 float high_freq_factor, float original_len, float* table, void* stream);

/* The q/k/v projections of a decode step in one launch, with the attention
 * norm folded in (as qmatmul_gemv_grouped_rmsnorm) and RoPE plus the cache
 * append as the GEMV epilogue (Sec. 3.3: each fusion removes a launch).
 * w: three descriptors, q [n_q_heads * head_dim][k], k and v
 * [n_kv_heads * head_dim][k], one format (any of the eight), DEVICE layout; the rows of each
 * head of w[0] and w[1] are stored interleaved: stored row 2i is the head's
 * row i and stored row 2i + 1 its row i + head_dim/2 (so a rotation pair is
 * computed by neighbouring lanes).  Writes q_out (fp16 [n_q_heads][head_dim],
 * rotated, in the natural order), row pos of k_cache (rotated) and of
 * v_cache (fp16 [n_kv_heads][max_len][head_dim]) and x_out; rope_table from
 * qdec_rope_table for this max_len and head_dim.  x, residual, gain, eps,
 * x_out as qmatmul_gemv_grouped_rmsnorm. */
qm_status qmatmul_gemv_qkv_rmsnorm_rope(const qm_qweight* w, const float* x, const float* residual,
                                        const uint16_t* gain, float eps, float* x_out, int32_t n_q_heads,
                                        int32_t n_kv_heads, int32_t head_dim, int64_t pos, int64_t max_len,
                                        const float* rope_table, uint16_t* q_out, uint16_t* k_cache,
                                        uint16_t* v_cache, void* stream);

/* Grouped decode GEMV (Sec. 3.3: fusing a sequence of operators removes a
 * launch each, which matters most in decode; e.g. the q/k/v projections of
 * a layer, which share x, or its gate and up projections):
 *   y_i[n] = sum_k s_i[n][k/32] * q_i[n][k] * x_i[k]   for i < count,
 * in one launch when the group's total rows stay below 64 rows per CU (else
 * one launch per matrix).  w: host array of `count` descriptors, all DEVICE
 * layout, batch 1, one format and one k; n_i may differ.  x, y: host arrays
 * of `count` device pointers; x_i fp16 [k], 16-byte aligned, and may be
 * shared between entries; y_i fp32 [n_i], 4-byte aligned, must not overlap
 * each other or any x_i.  1 <= count <= 8 (QM_GEMV_GROUP_MAX).  Same
 * arithmetic as qmatmul_gemv (the summation order may differ, since the
 * launch plan follows the group's total rows).  No workspace, deterministic. */
#define QM_GEMV_GROUP_MAX 8
qm_status qmatmul_gemv_grouped(int32_t count, const qm_qweight* w, const uint16_t* const* x,
                               float* const* y, void* stream);

/* Grouped prefill GEMM (Sec. 3.3: each fusion removes a launch; e.g. the
 * q/k/v projections of a layer, or its gate and up projections, which all
 * read the same X):  Y_i[m][n_i] = sum_k X[m][k] * w_i'[n_i][k]  for
 * i < count, in one launch.  w: host array of `count` descriptors, all of
 * one format (any of the eight), DEVICE layout, batch 1,
 * one k; n_i may differ.  X: fp16 [m][k] row-major
 * (device, 16-byte aligned), shared by all entries.  y: host array of
 * `count` device pointers to fp32 [m][n_i], 4-byte aligned, not
 * overlapping.  1 <= count <= 4 (QM_GEMM_GROUP_MAX); 1 <= m <= 65536 (m == 1
 * runs the grouped GEMV).  Same arithmetic as qmatmul_gemm per entry (the
 * split-K partition may differ, since the tile plan follows the group's
 * total columns).  Deterministic. */
#define QM_GEMM_GROUP_MAX 4
qm_status qmatmul_gemm_grouped(int32_t count, const qm_qweight* w, const uint16_t* x, int64_t m,
                               float* const* y, void* stream);

/* Prefill GEMM (Sec. 3.3, Sec. 3.4, M > 1): Y[m][n] = sum_k X[m][k] * w'[n][k].
 * w: DEVICE layout, batch 1, any of the eight formats of Sec. 4.1 (one MFMA
 * path; only the in-register unpacking differs).
 * X: fp16 [m][k] row-major; Y: fp32 [m][n].
 * X tiles and (for most tile shapes) the raw weight chunks are copied into
 * LDS by DMA; integer-format weights are dequantised to fp16 (value
 * fp16_RNE(s*q)) in registers, F16 weights are used as stored and BF16
 * weights are converted to fp16 (exact for |w| in [2^-14, 65504]; smaller
 * magnitudes round to fp16 subnormals, larger ones overflow to inf), all fed
 * to fp16 MFMA with fp32 accumulation.
 * m >= 1 (m == 1 runs the GEMV); m <= 65536 per call (chunk larger
 * prompts).  Deterministic. */
qm_status qmatmul_gemm(const qm_qweight* w, const uint16_t* x, int64_t m, float* y, void* stream);

/* Causal prefill attention over a prompt chunk (Sec. 3.4: FlashAttention,
 * key blocks folded in one at a time while each query row carries its running
 * maximum and sum, so memory grows linearly with the chunk; chunks of bounded
 * size):
 *   o[h][i] = sum_{j <= p0 + i} p_j v[g][j],  p = softmax_j(scale * q[h][i] . k[g][j]),
 *   g = h / (n_q_heads / n_kv_heads),  i < m.
 * q: fp16 [n_q_heads][m][head_dim], the chunk's queries at positions p0 ..
 * p0 + m - 1; k_cache, v_cache: fp16 [n_kv_heads][max_len][head_dim] holding
 * positions 0 .. p0 + m - 1 (the chunk's own keys and values written
 * already); o: fp32 [n_q_heads][m][head_dim]; q, the caches, o and the
 * workspace 16-byte aligned.  head_dim 64 or 128;
 * 1 <= m <= 65536; p0 + m <= max_len <= 262144; scale finite and > 0.
 * fp16 MFMA for q.k and p.v (p rounded toward zero to fp16; the sums use
 * the fp32 p), fp32 statistics and accumulation.
 * workspace (device, 16-byte aligned, or NULL): long query tiles of the
 * causal triangle are split over key ranges whose partial sums, maxima and
 * denominators go to the workspace and are merged by a second launch (the
 * online-softmax merge); qattn_prefill_workspace_bytes gives the bytes of
 * the full split plan on the current device.  A smaller workspace gives
 * fewer splits, NULL none (one launch).  Deterministic for a given
 * workspace size; calls sharing a workspace must not overlap. */
qm_status qattn_prefill(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t n_q_heads,
                        int32_t n_kv_heads, int32_t head_dim, int64_t m, int64_t p0, int64_t max_len, float scale,
                        float* o, void* workspace, size_t workspace_bytes, void* stream);

/* qattn_prefill with its output as the output projection's GEMM input:
 * out[i][h * head_dim + d] = fp16_RNE(o[h][i][d]), fp16 [m][n_q_heads *
 * head_dim] (16-byte aligned), the same values qattn_prefill followed by
 * qdec_heads_to_rows_f16 gives, written by the attention (and the merge)
 * itself.  (Sec. 3.4: chunked prefill; Sec. 3.3: the conversion fused into
 * the producing kernel, one launch fewer per layer.) */
qm_status qattn_prefill_rows_f16(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                 int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int64_t m, int64_t p0,
                                 int64_t max_len, float scale, uint16_t* out, void* workspace, size_t workspace_bytes,
                                 void* stream);

/* Bytes of qattn_prefill's workspace for its full key-split plan on the
 * current device (0 when no tile is split): per split range of a split
 * tile, n_q_heads x 128 rows x (head_dim + 4) floats.  Same shape limits as
 * qattn_prefill.  (Sec. 3.4: tiled attention; the key-range split is this
 * library's load balancing of the causal triangle.) */
qm_status qattn_prefill_workspace_bytes(int32_t n_q_heads, int32_t head_dim, int64_t m, int64_t p0, size_t* bytes);

/* Host-only: bytes of the decode-attention workspace for n_q_heads query
 * heads of head_dim (64 or 128): per query head up to 256 slices of
 * (head_dim + 2) floats.
 * (Sec. 3.2: caller-owned buffers, nothing allocated on the hot path.) */
qm_status qattn_decode_workspace_bytes(int32_t n_q_heads, int32_t head_dim, size_t* bytes);

/* Decode attention over a pre-allocated KV cache (Sec. 3.2: the cache is
 * sized for the longest context up front, laid out for coalesced reads;
 * grouped-query attention as in the Llama 3.2 and Qwen3 models):
 *   o[h] = sum_t p_t v[g][t],  p = softmax_t(scale * q[h] . k[g][t]),
 *   g = h / (n_q_heads / n_kv_heads),  t < len.
 * q: fp16 [n_q_heads][head_dim]; k_cache, v_cache: fp16
 * [n_kv_heads][max_len][head_dim] (rows t >= len are not read as data);
 * o: fp32 [n_q_heads][head_dim].  head_dim 64 or 128; at most 8 query heads
 * per KV head; 1 <= len <= max_len <= 262144; scale finite.  q, k_cache,
 * v_cache, workspace 16-byte aligned; workspace of at least
 * qattn_decode_workspace_bytes() bytes (caller-owned scratch, contents not
 * preserved).  Scores and sums in fp32, split over the cache length and
 * merged exactly as online softmax does.  Two kernel launches (one, with no
 * merge, when len <= 128); deterministic. */
qm_status qattn_decode(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t n_q_heads,
                       int32_t n_kv_heads, int32_t head_dim, int64_t len, int64_t max_len, float scale, float* o,
                       void* workspace, size_t ws_bytes, void* stream);

/* As qattn_decode, with o written as fp16 [n_q_heads][head_dim] (round to
 * nearest even of the same fp32 value; 2-byte aligned), ready to be the
 * input of the output projection's GEMV.
 * (Sec. 3.3: the fp16 conversion fused into the producer.) */
qm_status qattn_decode_f16(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t n_q_heads,
                           int32_t n_kv_heads, int32_t head_dim, int64_t len, int64_t max_len, float scale,
                           uint16_t* o, void* workspace, size_t ws_bytes, void* stream);

/* ---- Glue of one decode step (Sec. 3.2: the normalisation, RoPE,
 * embedding and sampling kernels between the matmuls and attention of a
 * dense Llama 3.2 / Qwen3-style decoder).  Activations handed to a matmul or
 * to attention are fp16; the residual stream is fp32.  None of these entry
 * points synchronises with the host: with the token id on the device, one
 * step's argmax feeds the next step's embedding. */

/* x[i] = table[*token][i] (fp16 -> fp32), i < hidden.  table: fp16
 * [vocab][hidden]; token: one int32 on the device; an id outside
 * [0, vocab) writes NaNs into x (a host check would need a synchronisation).
 * (Sec. 3.2: embedding kernel of the decode step.) */
qm_status qdec_embed(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* token, float* x,
                     void* stream);

/* RMSNorm of `rows` rows of x (fp32 [rows][hidden], device), with an
 * optional residual add first:  if residual != NULL, x += residual (written
 * back into x);  out = fp16_RNE(x / sqrt(mean(x^2) + eps) * w).  w: fp16
 * [hidden]; out: fp16 [rows][hidden].  Sum of squares in fp32.  rows may be
 * 0; hidden >= 1; eps finite and >= 0.
 * (Sec. 3.2: normalisation kernel of the decode step.) */
qm_status qdec_rmsnorm(float* x, const float* residual, const uint16_t* w, int64_t rows, int64_t hidden, float eps,
                       uint16_t* out, void* stream);

/* Rotary embedding of the new token's queries and keys, fused with the
 * KV-cache append (rotate-half pairing: element i with i + head_dim/2,
 * angle pos * theta^(-2i/head_dim), taken in fp64):
 *   q_out[h] = fp16(rope(q[h]))          h < n_q_heads,
 *   k_cache[g][pos] = fp16(rope(k[g])),  v_cache[g][pos] = fp16(v[g]).
 * q: fp32 [n_q_heads][head_dim]; k, v: fp32 [n_kv_heads][head_dim] (the
 * projection outputs); q_out: fp16 [n_q_heads][head_dim]; caches: fp16
 * [n_kv_heads][max_len][head_dim], only row pos of each head written.
 * head_dim 64 or 128; 0 <= pos < max_len <= 262144; theta > 1.
 * q_norm, k_norm: fp16 [head_dim] gains of the per-head RMSNorm the Qwen3
 * layer applies to every query and key head before RoPE
 * (x / sqrt(mean over the head(x^2) + eps) * gain, sum in fp32); both NULL
 * for the Llama layer.
 * table: NULL, or qdec_rope_table's (cos, sin) pairs for this head_dim and
 * theta over table_len > pos positions (8-byte aligned), read instead of
 * computing the angles (the same values).
 * (Sec. 3.2: RoPE and the KV cache of the decode step.) */
qm_status qdec_rope_append(const float* q, const float* k, const float* v, int32_t n_q_heads, int32_t n_kv_heads,
                           int32_t head_dim, int64_t pos, int64_t max_len, float theta, const uint16_t* q_norm,
                           const uint16_t* k_norm, float eps, const float* table, int64_t table_len,
                           uint16_t* q_out, uint16_t* k_cache, uint16_t* v_cache, void* stream);

/* out[i] = fp16_RNE(x[i]), i < n (values beyond the fp16 range become inf).
 * x: fp32, out: fp16, device; n >= 0.
 * (Sec. 3.2: conversion between the kernels of a decode step.) */
qm_status qdec_cast_f16(const float* x, int64_t n, uint16_t* out, void* stream);

/* Greedy sampling: *token = the index of the largest of logits[0 .. n),
 * the lowest index among equal maxima; NaNs are never chosen (0 if all
 * are NaN).  logits: fp32, device; token: one int32, device; n >= 1;
 * workspace: caller-owned device scratch of at least
 * QDEC_ARGMAX_WORKSPACE_BYTES bytes, 4-byte aligned, contents not
 * preserved (partial maxima of up to 256 workgroups).  One launch for
 * n <= 4096, else two.
 * (Sec. 3.2: sampling kernel of the decode step.) */
#define QDEC_ARGMAX_WORKSPACE_BYTES 2048
qm_status qdec_argmax(const float* logits, int64_t n, int32_t* token, void* workspace, size_t ws_bytes,
                      void* stream);

/* Host-only: workspace bytes qmoe_grouped_gemm needs for m tokens, so the
 * caller allocates it once for the largest chunk (Sec. 3.2: no allocation on
 * the hot path; Sec. 3.4: bounded prefill chunks).  Covers h and the
 * per-assignment outputs. */
qm_status qmoe_workspace_bytes(int64_t m, int32_t n_experts, int32_t top_k, int64_t hidden,
                               int64_t inter, size_t* bytes);

/* MoE routing and bucketing for the mixture-of-experts models (Sec. 4.1:
 * Qwen3-30B-A3B, 128 experts, 8 active per token; the paper gives no routing
 * formula, so the top-k-then-softmax router of the model family is taken)
 * (device in/out; all int32/fp32):
 *  logits [m][n_experts] fp32 -> topk_ids [m][top_k]: per token the top_k
 *  experts by logit, descending, equal logits -> lower expert first;
 *  topk_w [m][top_k]: softmax over those top_k logits (fp32);
 *  counts [n_experts], offsets [n_experts + 1] (exclusive prefix sum,
 *  offsets[E] = m*top_k) and sorted_assign [m*top_k]: the flat assignment
 *  ids a = t*top_k + j grouped by expert, ascending a inside each expert
 *  (stable counting sort).  n_experts <= 1024, 1 <= top_k <= min(16, n_experts),
 *  m <= 65536.  Ids, counts, offsets and sorted_assign are deterministic. */
qm_status qmoe_route(const float* logits, int64_t m, int32_t n_experts, int32_t top_k,
                     int32_t* topk_ids, float* topk_w, int32_t* counts, int32_t* offsets,
                     int32_t* sorted_assign, void* stream);

/* Routed SwiGLU expert layer (grouped GEMMs + weighted combine) of the MoE
 * models (Sec. 4.1; Sec. 3.3: the quantised GEMM per format with the
 * activation fused into the producing kernel; Sec. 4.3: MoE prefill):
 *  for every assignment a = t*top_k + j, with e the expert whose bucket
 *  [offsets[e], offsets[e+1]) of sorted_assign holds a:
 *    h_a = silu(Wg_e x_t) * (Wu_e x_t),  y_a = Wd_e h_a,
 *  y[t] = sum_j topk_w[t][j] * y_{t*top_k+j}, summed in slot order j.
 *  w_gate, w_up: DEVICE layout, batch E, [E][inter][hidden];
 *  w_down: DEVICE layout, batch E, [E][hidden][inter]; all three in one of
 *  Q2, Q3, Q4, Q5, Q6, Q8 (QM_EFORMAT if they differ, or for F16 / BF16);
 *  x: fp16 [m][hidden]; y: fp32 [m][hidden]; topk_ids, topk_w [m][top_k],
 *  counts, offsets and sorted_assign come from qmoe_route (sorted_assign
 *  must be a permutation of 0 .. m*top_k-1 consistent with counts/offsets).
 *  topk_ids is checked on the device against the buckets: an assignment a
 *  placed in the bucket of expert e with topk_ids[a] != e makes its token's
 *  row of y NaN (no host synchronisation, so no status code for it).
 *  hidden % 32 == 0 and inter % 32 == 0.  h and the gate-weighted
 *  per-assignment outputs topk_w * y_a are held in fp16 (summed in fp32);
 *  all GEMMs use fp16 MFMA with fp32 accumulation.  The workspace (device,
 *  16-byte aligned, >= qmoe_workspace_bytes) holds h and the per-assignment
 *  outputs; no host synchronisation: per-expert row counts stay on the
 *  device.  Deterministic. */
qm_status qmoe_grouped_gemm(const qm_qweight* w_gate, const qm_qweight* w_up,
                            const qm_qweight* w_down, const uint16_t* x, int64_t m,
                            int32_t top_k, const int32_t* topk_ids, const float* topk_w,
                            const int32_t* counts, const int32_t* offsets,
                            const int32_t* sorted_assign, float* y, void* workspace,
                            size_t ws_bytes, void* stream);

/* qmoe_grouped_gemm for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * kernels and results, with h and the per-assignment outputs in a scratch
 * array the library holds in device memory (QMOE_NOALLOC_SCRATCH_BYTES per
 * device, kept by every device the library runs on until the process ends)
 * instead of a caller workspace.  Allocates nothing and calls no allocating
 * routine.  Arguments as qmoe_grouped_gemm; QM_EWORKSPACE when the layer
 * needs more than QMOE_NOALLOC_SCRATCH_BYTES (qmoe_workspace_bytes tells:
 * e.g. up to 744 tokens at top-8, hidden 2048, inter 768).  Every call on a
 * device uses the same scratch: calls that overlap on one device (other
 * streams, other threads) race; order them on one stream. */
#define QMOE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
qm_status qmoe_grouped_gemm_noalloc(const qm_qweight* w_gate, const qm_qweight* w_up,
                                    const qm_qweight* w_down, const uint16_t* x, int64_t m,
                                    int32_t top_k, const int32_t* topk_ids, const float* topk_w,
                                    const int32_t* counts, const int32_t* offsets,
                                    const int32_t* sorted_assign, float* y, void* stream);

/* Writes a one-line description of the per-chip launch table chosen for the
 * current device into buf (Sec. 3.3: kernel geometry from a per-chip
 * configuration): arch, CU count, the Q4 GEMV kernel (name with template
 * arguments) of each projection shape of the benchmark decode stacks as
 * "gemv_q4(K->N)=name", and the prefill and MoE tile choices.  Truncated
 * to len - 1 characters (about 1 KiB is enough). */
qm_status qm_device_config(char* buf, size_t len);

#ifdef __cplusplus
}
#endif

#endif /* QMATMUL_H */
