// C ABI entry points: argument validation (nothing is enqueued on error),
// the thread-local error buffer, the per-device configuration and dispatch
// to the kernel launchers.
//
// The library allocates nothing and keeps no per-call state (BaseRT Sec. 3.2:
// no memory is requested on the decode path once a model is loaded, and error
// text lives in a fixed per-thread buffer); the only shared state is an
// immutable per-device table (CU count, architecture) built once per device.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "qm_internal.h"

namespace qm {
namespace {

thread_local char g_err[512] = "";

struct DeviceInfo {
  int cu_count = 0;
  char arch[64] = "";
  hipError_t status = hipSuccess;
};

constexpr int kMaxDevices = 64;
DeviceInfo g_dev[kMaxDevices];
std::once_flag g_dev_once[kMaxDevices];

qm_status device_info(const DeviceInfo** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(QM_EDEVICE, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(QM_EDEVICE, "device index %d out of range", dev);
  std::call_once(g_dev_once[dev], [dev]() {
    DeviceInfo& d = g_dev[dev];
    hipDeviceProp_t prop;
    d.status = hipGetDeviceProperties(&prop, dev);
    if (d.status == hipSuccess) {
      d.cu_count = prop.multiProcessorCount;
      std::snprintf(d.arch, sizeof(d.arch), "%s", prop.gcnArchName);
    }
  });
  const DeviceInfo& d = g_dev[dev];
  if (d.status != hipSuccess)
    return fail(QM_EDEVICE, "hipGetDeviceProperties failed: %s", hipGetErrorString(d.status));
  if (std::strncmp(d.arch, "gfx950", 6) != 0)
    return fail(QM_EDEVICE, "device %d is %s; this library is built for gfx950 only", dev, d.arch);
  *out = &d;
  return QM_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }
bool aligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }
bool aligned2(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 1u) == 0; }

qm_status check_weight(const qm_qweight* w, const char* name) {
  if (!w) return fail(QM_EINVAL, "%s: null weight descriptor", name);
  if (!fmt_valid(w->format)) return fail(QM_EFORMAT, "%s: unknown format %d", name, w->format);
  if (w->layout != QM_LAYOUT_CANONICAL && w->layout != QM_LAYOUT_DEVICE)
    return fail(QM_ELAYOUT, "%s: unknown layout %d", name, w->layout);
  if (w->batch < 1 || w->n < 0 || w->k < 0)
    return fail(QM_ESHAPE, "%s: bad shape batch=%lld n=%lld k=%lld", name, (long long)w->batch,
                (long long)w->n, (long long)w->k);
  if (w->k % kGroup != 0 || w->k == 0)
    return fail(QM_ESHAPE, "%s: k=%lld must be a positive multiple of 32", name, (long long)w->k);
  if (w->n >= (int64_t(1) << 31) || w->k >= (int64_t(1) << 31))
    return fail(QM_ESHAPE, "%s: n and k must be < 2^31", name);
  const bool scaled = !fmt_float(w->format);
  if (w->n > 0 && (!w->qdata || (scaled && !w->scales))) return fail(QM_EINVAL, "%s: null data pointer", name);
  if (!aligned16(w->qdata) || (scaled && !aligned16(w->scales)))
    return fail(QM_EALIGN, "%s: qdata and scales must be 16-byte aligned", name);
  return QM_OK;
}

}  // namespace

qm_status fail(qm_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

qm_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(QM_EDEVICE, "%s: launch failed: %s", what, hipGetErrorString(e));
  return QM_OK;
}

static qm_status launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(QM_EDEVICE, "%s: launch failed: %s", what, hipGetErrorString(e));
  return QM_OK;
}

}  // namespace qm

using namespace qm;

extern "C" {

const char* qm_last_error(void) { return g_err; }

qm_status qm_weight_bytes(int32_t format, int32_t layout, int64_t batch, int64_t n, int64_t k,
                          size_t* qbytes, size_t* sbytes) {
  if (!qbytes || !sbytes) return fail(QM_EINVAL, "qm_weight_bytes: null output pointer");
  if (!fmt_valid(format)) return fail(QM_EFORMAT, "qm_weight_bytes: unknown format %d", format);
  if (layout != QM_LAYOUT_CANONICAL && layout != QM_LAYOUT_DEVICE)
    return fail(QM_ELAYOUT, "qm_weight_bytes: unknown layout %d", layout);
  if (batch < 1 || n < 0 || k <= 0 || k % kGroup != 0)
    return fail(QM_ESHAPE, "qm_weight_bytes: bad shape batch=%lld n=%lld k=%lld", (long long)batch,
                (long long)n, (long long)k);
  const int64_t rows = batch * matrix_rows(layout, n);
  *qbytes = static_cast<size_t>(rows * row_code_bytes(format, k));
  *sbytes = static_cast<size_t>(rows * row_scales(format, k) * 2);
  return QM_OK;
}

qm_status qm_quantise(int32_t format, const float* w, const qm_qweight* out, void* stream) {
  qm_status st = check_weight(out, "qm_quantise(out)");
  if (st != QM_OK) return st;
  if (out->format != format)
    return fail(QM_EFORMAT, "qm_quantise: out->format %d != format %d", out->format, format);
  if (out->layout != QM_LAYOUT_CANONICAL)
    return fail(QM_ELAYOUT, "qm_quantise: output must be in CANONICAL layout");
  if (out->n > 0 && !w) return fail(QM_EINVAL, "qm_quantise: null input");
  if (!aligned16(w)) return fail(QM_EALIGN, "qm_quantise: w must be 16-byte aligned");
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_quantise(format, w, static_cast<uint8_t*>(out->qdata), out->scales, out->batch,
                                  out->n, out->k, static_cast<hipStream_t>(stream)),
                  "qm_quantise");
}

qm_status qm_dequantise(const qm_qweight* w, float* out, void* stream) {
  qm_status st = check_weight(w, "qm_dequantise(w)");
  if (st != QM_OK) return st;
  if (w->n > 0 && !out) return fail(QM_EINVAL, "qm_dequantise: null output");
  if (!aligned16(out)) return fail(QM_EALIGN, "qm_dequantise: out must be 16-byte aligned");
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_dequantise(w->format, w->layout, static_cast<const uint8_t*>(w->qdata),
                                    w->scales, out, w->batch, w->n, w->k,
                                    static_cast<hipStream_t>(stream)),
                  "qm_dequantise");
}

qm_status qm_repack(const qm_qweight* src, const qm_qweight* dst, void* stream) {
  qm_status st = check_weight(src, "qm_repack(src)");
  if (st != QM_OK) return st;
  if ((st = check_weight(dst, "qm_repack(dst)")) != QM_OK) return st;
  if (src->format != dst->format) return fail(QM_EFORMAT, "qm_repack: formats differ");
  if (src->layout == dst->layout) return fail(QM_ELAYOUT, "qm_repack: src and dst layouts are equal");
  if (src->batch != dst->batch || src->n != dst->n || src->k != dst->k)
    return fail(QM_ESHAPE, "qm_repack: shapes differ");
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_repack(src->format, src->layout, static_cast<const uint8_t*>(src->qdata),
                                src->scales, static_cast<uint8_t*>(dst->qdata), dst->scales, src->batch,
                                src->n, src->k, static_cast<hipStream_t>(stream)),
                  "qm_repack");
}

qm_status qmatmul_gemv(const qm_qweight* w, const uint16_t* x, float* y, void* stream) {
  qm_status st = check_weight(w, "qmatmul_gemv(w)");
  if (st != QM_OK) return st;
  if (w->layout != QM_LAYOUT_DEVICE) return fail(QM_ELAYOUT, "qmatmul_gemv: weights must be in DEVICE layout");
  if (w->batch != 1) return fail(QM_ESHAPE, "qmatmul_gemv: batch must be 1");
  if (w->n > 0 && (!x || !y)) return fail(QM_EINVAL, "qmatmul_gemv: null x or y");
  if (!aligned16(x)) return fail(QM_EALIGN, "qmatmul_gemv: x must be 16-byte aligned");
  if (!aligned4(y)) return fail(QM_EALIGN, "qmatmul_gemv: y must be 4-byte aligned");
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_gemv(w->format, static_cast<const uint8_t*>(w->qdata), w->scales, x, y, w->n,
                              w->k, d->cu_count, static_cast<hipStream_t>(stream)),
                  "qmatmul_gemv");
}

}  // extern "C"

namespace {

// Shared checks and launch of the SwiGLU pair; out is h (fp32) or h16 (fp16).
qm_status swiglu_call(const qm_qweight* w_gate, const qm_qweight* w_up, const uint16_t* x, float* h, uint16_t* h16,
                      void* stream, const char* name) {
  char what[64];
  std::snprintf(what, sizeof(what), "%s(w_gate)", name);
  qm_status st = check_weight(w_gate, what);
  if (st != QM_OK) return st;
  std::snprintf(what, sizeof(what), "%s(w_up)", name);
  if ((st = check_weight(w_up, what)) != QM_OK) return st;
  if (w_gate->layout != QM_LAYOUT_DEVICE || w_up->layout != QM_LAYOUT_DEVICE)
    return fail(QM_ELAYOUT, "%s: weights must be in DEVICE layout", name);
  if (w_gate->batch != 1 || w_up->batch != 1) return fail(QM_ESHAPE, "%s: batch must be 1", name);
  if (w_up->format != w_gate->format) return fail(QM_EFORMAT, "%s: formats differ", name);
  if (w_up->n != w_gate->n || w_up->k != w_gate->k) return fail(QM_ESHAPE, "%s: gate and up shapes differ", name);
  if (w_gate->n > INT32_MAX / 2) return fail(QM_ESHAPE, "%s: n too large", name);
  if (w_gate->n > 0 && (!x || (!h && !h16))) return fail(QM_EINVAL, "%s: null x or h", name);
  if (!aligned16(x)) return fail(QM_EALIGN, "%s: x must be 16-byte aligned", name);
  if (!aligned4(h) || !aligned2(h16)) return fail(QM_EALIGN, "%s: h must be 4-byte (fp32) or 2-byte (fp16) aligned", name);
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_gemv_swiglu(w_gate->format, static_cast<const uint8_t*>(w_gate->qdata), w_gate->scales,
                                     static_cast<const uint8_t*>(w_up->qdata), w_up->scales, x, h, h16, w_gate->n,
                                     w_gate->k, d->cu_count, static_cast<hipStream_t>(stream)),
                  name);
}

}  // namespace

extern "C" {

qm_status qmatmul_gemv_swiglu(const qm_qweight* w_gate, const qm_qweight* w_up, const uint16_t* x, float* h,
                              void* stream) {
  return swiglu_call(w_gate, w_up, x, h, nullptr, stream, "qmatmul_gemv_swiglu");
}

qm_status qmatmul_gemv_swiglu_f16(const qm_qweight* w_gate, const qm_qweight* w_up, const uint16_t* x, uint16_t* h,
                                  void* stream) {
  return swiglu_call(w_gate, w_up, x, nullptr, h, stream, "qmatmul_gemv_swiglu_f16");
}

}  // extern "C"

namespace {

// Checks of the fused-RMSNorm inputs shared by the two fused entry points.
qm_status check_norm(const float* x, const float* residual, const uint16_t* gain, float eps, const float* x_out,
                     int64_t k, const char* name) {
  if (k > kNormGemvMaxK) return fail(QM_ESHAPE, "%s: k=%lld must be <= %lld", name, (long long)k,
                                     (long long)kNormGemvMaxK);
  if (!(eps >= 0.0f) || eps == INFINITY) return fail(QM_EINVAL, "%s: eps must be finite and >= 0", name);
  if (!x || !gain || !x_out) return fail(QM_EINVAL, "%s: null x, gain or x_out", name);
  if (!aligned16(x) || !aligned16(residual) || !aligned16(x_out) ||
      (reinterpret_cast<uintptr_t>(gain) & 7u) != 0)
    return fail(QM_EALIGN, "%s: x, residual and x_out must be 16-byte aligned, gain 8-byte aligned", name);
  const uintptr_t o0 = reinterpret_cast<uintptr_t>(x_out), o1 = o0 + static_cast<uintptr_t>(k) * 4;
  auto overlaps = [&](const void* p) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(p), a1 = a0 + static_cast<uintptr_t>(k) * 4;
    return p && a0 < o1 && o0 < a1;
  };
  if (overlaps(x) || overlaps(residual)) return fail(QM_EINVAL, "%s: x_out must not overlap x or residual", name);
  return QM_OK;
}

}  // namespace

extern "C" {

qm_status qmatmul_gemv_grouped_rmsnorm(int32_t count, const qm_qweight* w, const float* x, const float* residual,
                                       const uint16_t* gain, float eps, float* x_out, float* const* y,
                                       void* stream) {
  const char* name = "qmatmul_gemv_grouped_rmsnorm";
  if (count < 1 || count > QM_GEMV_GROUP_MAX)
    return fail(QM_ESHAPE, "%s: count=%d must be in [1, %d]", name, count, QM_GEMV_GROUP_MAX);
  if (!w || !y) return fail(QM_EINVAL, "%s: null array", name);
  GemvGroup g{};
  g.count = count;
  for (int i = 0; i < count; ++i) {
    qm_status st = check_weight(&w[i], "qmatmul_gemv_grouped_rmsnorm(w[i])");
    if (st != QM_OK) return st;
    if (w[i].layout != QM_LAYOUT_DEVICE) return fail(QM_ELAYOUT, "%s: w[%d] must be in DEVICE layout", name, i);
    if (w[i].batch != 1) return fail(QM_ESHAPE, "%s: w[%d] batch must be 1", name, i);
    if (w[i].format != w[0].format) return fail(QM_EFORMAT, "%s: formats differ", name);
    if (w[i].k != w[0].k) return fail(QM_ESHAPE, "%s: k differs between entries", name);
    if (w[i].n < 1 || w[i].n > INT32_MAX / 2) return fail(QM_ESHAPE, "%s: n of w[%d] must be in [1, 2^30]", name, i);
    if (!y[i]) return fail(QM_EINVAL, "%s: null y[%d]", name, i);
    if (!aligned4(y[i])) return fail(QM_EALIGN, "%s: y[%d] must be 4-byte aligned", name, i);
    g.q[i] = static_cast<const uint8_t*>(w[i].qdata);
    g.s[i] = w[i].scales;
    g.y[i] = y[i];
    g.n[i] = static_cast<int>(w[i].n);
  }
  qm_status st = check_norm(x, residual, gain, eps, x_out, w[0].k, name);
  if (st != QM_OK) return st;
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  const NormArgs na{x, residual, gain, x_out, eps};
  return launched(launch_gemv_group_norm(w[0].format, g, na, w[0].k, d->cu_count, static_cast<hipStream_t>(stream)),
                  name);
}

qm_status qdec_embed_rows(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* tokens, int64_t m,
                          float* x, void* stream) {
  if (vocab < 1 || vocab > INT32_MAX || hidden < 1 || hidden > (int64_t{1} << 20) || m < 0 || m > 32768)
    return fail(QM_ESHAPE, "qdec_embed_rows: need 1 <= vocab < 2^31, 1 <= hidden <= 2^20, 0 <= m <= 32768");
  if (m > 0 && (!table || !tokens || !x)) return fail(QM_EINVAL, "qdec_embed_rows: null pointer");
  if (!aligned2(table) || !aligned4(tokens) || !aligned4(x))
    return fail(QM_EALIGN, "qdec_embed_rows: table 2-byte, tokens and x 4-byte aligned");
  return launched(launch_embed_rows(table, vocab, hidden, tokens, m, x, static_cast<hipStream_t>(stream)),
                  "qdec_embed_rows");
}

qm_status qdec_rope_append_rows(const float* q, const float* k, const float* v, int32_t n_q_heads,
                                int32_t n_kv_heads, int32_t head_dim, int64_t m, int64_t p0, int64_t max_len,
                                float theta, int32_t interleaved, const uint16_t* q_norm, const uint16_t* k_norm,
                                float eps, const float* table, int64_t table_len, uint16_t* q_out,
                                uint16_t* k_cache, uint16_t* v_cache, void* stream) {
  const char* name = "qdec_rope_append_rows";
  if (table && (!aligned8(table) || table_len < p0 + m))
    return fail(QM_EINVAL, "%s: the (cos, sin) table must be 8-byte aligned and cover positions < p0 + m", name);
  if ((q_norm == nullptr) != (k_norm == nullptr) || !aligned2(q_norm) || !aligned2(k_norm))
    return fail(QM_EINVAL, "%s: q_norm and k_norm both given (2-byte aligned) or both NULL", name);
  if (q_norm && (!(eps >= 0.0f) || eps == INFINITY)) return fail(QM_EINVAL, "%s: eps finite and >= 0", name);
  if (head_dim != 64 && head_dim != 128) return fail(QM_ESHAPE, "%s: head_dim=%d must be 64 or 128", name, head_dim);
  if (n_q_heads < 1 || n_q_heads > 1024 || n_kv_heads < 1 || n_kv_heads > 1024)
    return fail(QM_ESHAPE, "%s: head counts must be in [1, 1024]", name);
  if (m < 1 || m > 32768 || p0 < 0 || max_len > kAttnMaxLen || p0 + m > max_len)
    return fail(QM_ESHAPE, "%s: need 1 <= m <= 32768, p0 >= 0, p0 + m <= max_len <= %lld", name,
                (long long)kAttnMaxLen);
  if (!(theta > 1.0f) || theta == INFINITY) return fail(QM_EINVAL, "%s: theta must be finite and > 1", name);
  if (interleaved != 0 && interleaved != 1) return fail(QM_EINVAL, "%s: interleaved must be 0 or 1", name);
  if (!q || !k || !v || !q_out || !k_cache || !v_cache) return fail(QM_EINVAL, "%s: null pointer", name);
  if (!aligned4(q) || !aligned4(k) || !aligned4(v) || !aligned2(q_out) || !aligned2(k_cache) || !aligned2(v_cache))
    return fail(QM_EALIGN, "%s: q, k, v 4-byte, q_out and caches 2-byte aligned", name);
  return launched(launch_rope_append_rows(q, k, v, n_q_heads, n_kv_heads, head_dim, m, p0, max_len, theta,
                                          interleaved, q_out, k_cache, v_cache, q_norm, k_norm, eps, table,
                                          static_cast<hipStream_t>(stream)),
                  name);
}

qm_status qdec_heads_to_rows_f16(const float* o, int32_t n_heads, int64_t m, int32_t head_dim, uint16_t* out,
                                 void* stream) {
  if (n_heads < 1 || n_heads > 1024 || m < 1 || m > 65536 || head_dim < 1 || head_dim > 256)
    return fail(QM_ESHAPE, "qdec_heads_to_rows_f16: need 1 <= n_heads <= 1024, 1 <= m <= 65536, 1 <= head_dim <= 256");
  if (!o || !out) return fail(QM_EINVAL, "qdec_heads_to_rows_f16: null pointer");
  if (!aligned4(o) || !aligned2(out)) return fail(QM_EALIGN, "qdec_heads_to_rows_f16: o 4-byte, out 2-byte aligned");
  return launched(launch_heads_to_rows(o, n_heads, m, head_dim, out, static_cast<hipStream_t>(stream)),
                  "qdec_heads_to_rows_f16");
}

qm_status qdec_swiglu_f16(const float* gate, const float* up, int64_t n, uint16_t* out, void* stream) {
  if (n < 0) return fail(QM_ESHAPE, "qdec_swiglu_f16: n must be >= 0");
  if (n > 0 && (!gate || !up || !out)) return fail(QM_EINVAL, "qdec_swiglu_f16: null pointer");
  if (!aligned4(gate) || !aligned4(up) || !aligned2(out))
    return fail(QM_EALIGN, "qdec_swiglu_f16: gate and up 4-byte, out 2-byte aligned");
  return launched(launch_swiglu(gate, up, n, out, static_cast<hipStream_t>(stream)), "qdec_swiglu_f16");
}

qm_status qdec_rope_table(int64_t max_len, int32_t head_dim, float theta, float* table, void* stream) {
  if ((head_dim != 64 && head_dim != 128) || max_len < 1 || max_len > kAttnMaxLen)
    return fail(QM_ESHAPE, "qdec_rope_table: head_dim 64 or 128 and 1 <= max_len <= %lld", (long long)kAttnMaxLen);
  if (!(theta > 1.0f) || theta == INFINITY) return fail(QM_EINVAL, "qdec_rope_table: theta must be finite and > 1");
  if (!table) return fail(QM_EINVAL, "qdec_rope_table: null table");
  if ((reinterpret_cast<uintptr_t>(table) & 7u) != 0) return fail(QM_EALIGN, "qdec_rope_table: table 8-byte aligned");
  return launched(launch_rope_table(max_len, head_dim, theta, table, static_cast<hipStream_t>(stream)),
                  "qdec_rope_table");
}

qm_status qdec_rope_table_llama3(int64_t max_len, int32_t head_dim, float theta, float factor, float low_freq_factor,
                                 float high_freq_factor, float original_len, float* table, void* stream) {
  if ((head_dim != 64 && head_dim != 128) || max_len < 1 || max_len > kAttnMaxLen)
    return fail(QM_ESHAPE, "qdec_rope_table_llama3: head_dim 64 or 128 and 1 <= max_len <= %lld",
                (long long)kAttnMaxLen);
  if (!(theta > 1.0f) || theta == INFINITY) return fail(QM_EINVAL, "qdec_rope_table_llama3: theta must be finite and > 1");
  if (!(factor >= 1.0f) || factor == INFINITY || !(low_freq_factor > 0.0f) ||
      !(high_freq_factor > low_freq_factor) || high_freq_factor == INFINITY || !(original_len > 0.0f) ||
      original_len == INFINITY)
    return fail(QM_EINVAL, "qdec_rope_table_llama3: need finite factor >= 1, 0 < low_freq_factor < high_freq_factor "
                           "and original_len > 0");
  if (!table) return fail(QM_EINVAL, "qdec_rope_table_llama3: null table");
  if ((reinterpret_cast<uintptr_t>(table) & 7u) != 0)
    return fail(QM_EALIGN, "qdec_rope_table_llama3: table 8-byte aligned");
  return launched(launch_rope_table_llama3(max_len, head_dim, theta, factor, low_freq_factor, high_freq_factor,
                                           original_len, table, static_cast<hipStream_t>(stream)),
                  "qdec_rope_table_llama3");
}

qm_status qmatmul_gemv_qkv_rmsnorm_rope(const qm_qweight* w, const float* x, const float* residual,
                                        const uint16_t* gain, float eps, float* x_out, int32_t n_q_heads,
                                        int32_t n_kv_heads, int32_t head_dim, int64_t pos, int64_t max_len,
                                        const float* rope_table, uint16_t* q_out, uint16_t* k_cache,
                                        uint16_t* v_cache, void* stream) {
  const char* name = "qmatmul_gemv_qkv_rmsnorm_rope";
  if (!w) return fail(QM_EINVAL, "%s: null weights", name);
  if (head_dim != 64 && head_dim != 128) return fail(QM_ESHAPE, "%s: head_dim=%d must be 64 or 128", name, head_dim);
  if (n_q_heads < 1 || n_q_heads > 1024 || n_kv_heads < 1 || n_kv_heads > 1024)
    return fail(QM_ESHAPE, "%s: head counts must be in [1, 1024]", name);
  if (max_len < 1 || max_len > kAttnMaxLen || pos < 0 || pos >= max_len)
    return fail(QM_ESHAPE, "%s: need 0 <= pos < max_len <= %lld", name, (long long)kAttnMaxLen);
  const int64_t want[3] = {int64_t{n_q_heads} * head_dim, int64_t{n_kv_heads} * head_dim,
                           int64_t{n_kv_heads} * head_dim};
  GemvGroup g{};
  g.count = 3;
  for (int i = 0; i < 3; ++i) {
    qm_status st = check_weight(&w[i], "qmatmul_gemv_qkv_rmsnorm_rope(w[i])");
    if (st != QM_OK) return st;
    if (w[i].format != w[0].format) return fail(QM_EFORMAT, "%s: formats differ", name);
    if (w[i].layout != QM_LAYOUT_DEVICE) return fail(QM_ELAYOUT, "%s: w[%d] must be in DEVICE layout", name, i);
    if (w[i].batch != 1) return fail(QM_ESHAPE, "%s: w[%d] batch must be 1", name, i);
    if (w[i].k != w[0].k) return fail(QM_ESHAPE, "%s: k differs between entries", name);
    if (w[i].n != want[i]) return fail(QM_ESHAPE, "%s: w[%d] must have %lld rows", name, i, (long long)want[i]);
    g.q[i] = static_cast<const uint8_t*>(w[i].qdata);
    g.s[i] = w[i].scales;
    g.n[i] = static_cast<int>(w[i].n);
  }
  qm_status st = check_norm(x, residual, gain, eps, x_out, w[0].k, name);
  if (st != QM_OK) return st;
  if (!rope_table || !q_out || !k_cache || !v_cache) return fail(QM_EINVAL, "%s: null pointer", name);
  if ((reinterpret_cast<uintptr_t>(rope_table) & 7u) != 0 || !aligned2(q_out) || !aligned2(k_cache) ||
      !aligned2(v_cache))
    return fail(QM_EALIGN, "%s: rope_table 8-byte, q_out and caches 2-byte aligned", name);
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  const NormArgs na{x, residual, gain, x_out, eps};
  const QkvRopeEpi epi{q_out, k_cache, v_cache, rope_table, pos, max_len, head_dim};
  return launched(launch_gemv_qkv_norm_rope(w[0].format, g, na, epi, w[0].k, d->cu_count,
                                            static_cast<hipStream_t>(stream)),
                  name);
}

qm_status qmatmul_gemv_swiglu_rmsnorm_f16(const qm_qweight* w_gate, const qm_qweight* w_up, const float* x,
                                          const float* residual, const uint16_t* gain, float eps, float* x_out,
                                          uint16_t* h, void* stream) {
  const char* name = "qmatmul_gemv_swiglu_rmsnorm_f16";
  qm_status st = check_weight(w_gate, "qmatmul_gemv_swiglu_rmsnorm_f16(w_gate)");
  if (st != QM_OK) return st;
  if ((st = check_weight(w_up, "qmatmul_gemv_swiglu_rmsnorm_f16(w_up)")) != QM_OK) return st;
  if (w_gate->layout != QM_LAYOUT_DEVICE || w_up->layout != QM_LAYOUT_DEVICE)
    return fail(QM_ELAYOUT, "%s: weights must be in DEVICE layout", name);
  if (w_gate->batch != 1 || w_up->batch != 1) return fail(QM_ESHAPE, "%s: batch must be 1", name);
  if (w_up->format != w_gate->format) return fail(QM_EFORMAT, "%s: formats differ", name);
  if (w_up->n != w_gate->n || w_up->k != w_gate->k) return fail(QM_ESHAPE, "%s: gate and up shapes differ", name);
  if (w_gate->n < 1 || w_gate->n > INT32_MAX / 2) return fail(QM_ESHAPE, "%s: n must be in [1, 2^30]", name);
  if (!h) return fail(QM_EINVAL, "%s: null h", name);
  if (!aligned2(h)) return fail(QM_EALIGN, "%s: h must be 2-byte aligned", name);
  if ((st = check_norm(x, residual, gain, eps, x_out, w_gate->k, name)) != QM_OK) return st;
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  const NormArgs na{x, residual, gain, x_out, eps};
  return launched(launch_gemv_swiglu_norm(w_gate->format, static_cast<const uint8_t*>(w_gate->qdata), w_gate->scales,
                                          static_cast<const uint8_t*>(w_up->qdata), w_up->scales, na, nullptr, h,
                                          w_gate->n, w_gate->k, d->cu_count, static_cast<hipStream_t>(stream)),
                  name);
}

qm_status qmatmul_gemv_grouped(int32_t count, const qm_qweight* w, const uint16_t* const* x, float* const* y,
                               void* stream) {
  static_assert(QM_GEMV_GROUP_MAX == kGemvGroupMax, "group size");
  if (count < 1 || count > QM_GEMV_GROUP_MAX)
    return fail(QM_ESHAPE, "qmatmul_gemv_grouped: count=%d must be in [1, %d]", count, QM_GEMV_GROUP_MAX);
  if (!w || !x || !y) return fail(QM_EINVAL, "qmatmul_gemv_grouped: null array");
  GemvGroup g{};
  g.count = count;
  for (int i = 0; i < count; ++i) {
    qm_status st = check_weight(&w[i], "qmatmul_gemv_grouped(w[i])");
    if (st != QM_OK) return st;
    if (w[i].layout != QM_LAYOUT_DEVICE)
      return fail(QM_ELAYOUT, "qmatmul_gemv_grouped: w[%d] must be in DEVICE layout", i);
    if (w[i].batch != 1) return fail(QM_ESHAPE, "qmatmul_gemv_grouped: w[%d] batch must be 1", i);
    if (w[i].format != w[0].format) return fail(QM_EFORMAT, "qmatmul_gemv_grouped: formats differ");
    if (w[i].k != w[0].k) return fail(QM_ESHAPE, "qmatmul_gemv_grouped: k differs between entries");
    if (w[i].n > INT32_MAX / 2) return fail(QM_ESHAPE, "qmatmul_gemv_grouped: n too large");
    if (w[i].n > 0 && (!x[i] || !y[i])) return fail(QM_EINVAL, "qmatmul_gemv_grouped: null x[%d] or y[%d]", i, i);
    if (!aligned16(x[i])) return fail(QM_EALIGN, "qmatmul_gemv_grouped: x[%d] must be 16-byte aligned", i);
    if (!aligned4(y[i])) return fail(QM_EALIGN, "qmatmul_gemv_grouped: y[%d] must be 4-byte aligned", i);
    g.q[i] = static_cast<const uint8_t*>(w[i].qdata);
    g.s[i] = w[i].scales;
    g.x[i] = x[i];
    g.y[i] = y[i];
    g.n[i] = static_cast<int>(w[i].n);
  }
  const DeviceInfo* d;
  qm_status st;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_gemv_group(w[0].format, g, w[0].k, d->cu_count, static_cast<hipStream_t>(stream)),
                  "qmatmul_gemv_grouped");
}

qm_status qmatmul_gemm_grouped(int32_t count, const qm_qweight* w, const uint16_t* x, int64_t m, float* const* y,
                               void* stream) {
  static_assert(QM_GEMM_GROUP_MAX == kGemmGroupMax, "group size");
  if (count < 1 || count > QM_GEMM_GROUP_MAX)
    return fail(QM_ESHAPE, "qmatmul_gemm_grouped: count=%d must be in [1, %d]", count, QM_GEMM_GROUP_MAX);
  if (!w || !y) return fail(QM_EINVAL, "qmatmul_gemm_grouped: null array");
  if (m < 1 || m > 65536) return fail(QM_ESHAPE, "qmatmul_gemm_grouped: m=%lld must be in [1, 65536]", (long long)m);
  int64_t rows = 0;
  for (int i = 0; i < count; ++i) {
    qm_status st = check_weight(&w[i], "qmatmul_gemm_grouped(w[i])");
    if (st != QM_OK) return st;
    if (w[i].layout != QM_LAYOUT_DEVICE)
      return fail(QM_ELAYOUT, "qmatmul_gemm_grouped: w[%d] must be in DEVICE layout", i);
    if (w[i].batch != 1) return fail(QM_ESHAPE, "qmatmul_gemm_grouped: w[%d] batch must be 1", i);
    if (w[i].format != w[0].format) return fail(QM_EFORMAT, "qmatmul_gemm_grouped: formats differ");
    if (w[i].k != w[0].k) return fail(QM_ESHAPE, "qmatmul_gemm_grouped: k differs between entries");
    if (w[i].n > 0 && !y[i]) return fail(QM_EINVAL, "qmatmul_gemm_grouped: null y[%d]", i);
    if (!aligned4(y[i])) return fail(QM_EALIGN, "qmatmul_gemm_grouped: y[%d] must be 4-byte aligned", i);
    rows += padded_rows(w[i].n);
  }
  if (rows > (int64_t(1) << 30)) return fail(QM_ESHAPE, "qmatmul_gemm_grouped: too many rows in the group");
  if (rows > 0 && !x) return fail(QM_EINVAL, "qmatmul_gemm_grouped: null x");
  if (!aligned16(x)) return fail(QM_EALIGN, "qmatmul_gemm_grouped: x must be 16-byte aligned");
  const DeviceInfo* d;
  qm_status st;
  if ((st = device_info(&d)) != QM_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (m == 1) {
    GemvGroup g{};
    g.count = count;
    for (int i = 0; i < count; ++i) {
      g.q[i] = static_cast<const uint8_t*>(w[i].qdata); g.s[i] = w[i].scales;
      g.x[i] = x; g.y[i] = y[i]; g.n[i] = static_cast<int>(w[i].n);
    }
    return launched(launch_gemv_group(w[0].format, g, w[0].k, d->cu_count, s), "qmatmul_gemm_grouped(m=1)");
  }
  const uint8_t* qs[kGemmGroupMax];
  const uint16_t* ss[kGemmGroupMax];
  float* ys[kGemmGroupMax];
  int64_t ns[kGemmGroupMax];
  for (int i = 0; i < count; ++i) {
    qs[i] = static_cast<const uint8_t*>(w[i].qdata); ss[i] = w[i].scales; ys[i] = y[i]; ns[i] = w[i].n;
  }
  return launched(launch_gemm_group(w[0].format, count, qs, ss, ys, ns, x, m, w[0].k, d->cu_count, s),
                  "qmatmul_gemm_grouped");
}

qm_status qmatmul_gemm(const qm_qweight* w, const uint16_t* x, int64_t m, float* y, void* stream) {
  qm_status st = check_weight(w, "qmatmul_gemm(w)");
  if (st != QM_OK) return st;
  if (w->layout != QM_LAYOUT_DEVICE) return fail(QM_ELAYOUT, "qmatmul_gemm: weights must be in DEVICE layout");
  if (w->batch != 1) return fail(QM_ESHAPE, "qmatmul_gemm: batch must be 1");
  if (m < 1 || m > 65536) return fail(QM_ESHAPE, "qmatmul_gemm: m=%lld must be in [1, 65536]", (long long)m);
  if (w->n > 0 && (!x || !y)) return fail(QM_EINVAL, "qmatmul_gemm: null x or y");
  if (!aligned16(x)) return fail(QM_EALIGN, "qmatmul_gemm: x must be 16-byte aligned");
  if (!aligned4(y)) return fail(QM_EALIGN, "qmatmul_gemm: y must be 4-byte aligned");
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (m == 1)
    return launched(launch_gemv(w->format, static_cast<const uint8_t*>(w->qdata), w->scales, x, y, w->n,
                                w->k, d->cu_count, s),
                    "qmatmul_gemm(m=1)");
  return launched(launch_gemm(w->format, static_cast<const uint8_t*>(w->qdata), w->scales, x, y, m, w->n, w->k,
                              d->cu_count, s),
                  "qmatmul_gemm");
}

qm_status qattn_decode_workspace_bytes(int32_t n_q_heads, int32_t head_dim, size_t* bytes) {
  if (!bytes) return fail(QM_EINVAL, "qattn_decode_workspace_bytes: null output pointer");
  if (n_q_heads < 1 || n_q_heads > 1024 || (head_dim != 64 && head_dim != 128))
    return fail(QM_ESHAPE, "qattn_decode_workspace_bytes: n_q_heads in [1, 1024], head_dim 64 or 128");
  *bytes = attn_decode_workspace_bytes(n_q_heads, head_dim);
  return QM_OK;
}

}  // extern "C"

namespace {

// Shared checks and launch of decode attention; out is o (fp32) or o16 (fp16).
qm_status attn_decode_call(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t n_q_heads,
                           int32_t n_kv_heads, int32_t head_dim, int64_t len, int64_t max_len, float scale, float* o,
                           uint16_t* o16, void* workspace, size_t ws_bytes, void* stream, const char* name) {
  if (head_dim != 64 && head_dim != 128) return fail(QM_ESHAPE, "%s: head_dim=%d must be 64 or 128", name, head_dim);
  if (n_kv_heads < 1 || n_q_heads < 1 || n_q_heads > 1024 || n_q_heads % n_kv_heads != 0 ||
      n_q_heads / n_kv_heads > 8)
    return fail(QM_ESHAPE, "%s: n_q_heads=%d must be a multiple of n_kv_heads=%d, at most 8 per KV head", name,
                n_q_heads, n_kv_heads);
  if (max_len < 1 || max_len > kAttnMaxLen || len < 1 || len > max_len)
    return fail(QM_ESHAPE, "%s: need 1 <= len <= max_len <= %lld (len=%lld, max_len=%lld)", name,
                (long long)kAttnMaxLen, (long long)len, (long long)max_len);
  if (!(scale == scale) || scale == INFINITY || scale == -INFINITY)
    return fail(QM_EINVAL, "%s: scale must be finite", name);
  if (!q || !k_cache || !v_cache || (!o && !o16)) return fail(QM_EINVAL, "%s: null pointer", name);
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned4(o) || !aligned2(o16))
    return fail(QM_EALIGN, "%s: q, k_cache, v_cache must be 16-byte aligned, o 4-byte aligned", name);
  const size_t need = attn_decode_workspace_bytes(n_q_heads, head_dim);
  if (!workspace || ws_bytes < need)
    return fail(QM_EWORKSPACE, "%s: workspace of %zu bytes needed (got %zu)", name, need, ws_bytes);
  if (!aligned16(workspace)) return fail(QM_EALIGN, "%s: workspace must be 16-byte aligned", name);
  const DeviceInfo* d;
  qm_status st;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_attn_decode(q, k_cache, v_cache, n_q_heads, n_kv_heads, head_dim, len, max_len, scale, o, o16,
                                     static_cast<float*>(workspace), d->cu_count, static_cast<hipStream_t>(stream)),
                  name);
}

}  // namespace

extern "C" {

qm_status qattn_decode(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t n_q_heads,
                       int32_t n_kv_heads, int32_t head_dim, int64_t len, int64_t max_len, float scale, float* o,
                       void* workspace, size_t ws_bytes, void* stream) {
  return attn_decode_call(q, k_cache, v_cache, n_q_heads, n_kv_heads, head_dim, len, max_len, scale, o, nullptr,
                          workspace, ws_bytes, stream, "qattn_decode");
}

qm_status qattn_decode_f16(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t n_q_heads,
                           int32_t n_kv_heads, int32_t head_dim, int64_t len, int64_t max_len, float scale,
                           uint16_t* o, void* workspace, size_t ws_bytes, void* stream) {
  return attn_decode_call(q, k_cache, v_cache, n_q_heads, n_kv_heads, head_dim, len, max_len, scale, nullptr, o,
                          workspace, ws_bytes, stream, "qattn_decode_f16");
}

qm_status qattn_prefill_workspace_bytes(int32_t n_q_heads, int32_t head_dim, int64_t m, int64_t p0, size_t* bytes) {
  if (!bytes) return fail(QM_EINVAL, "qattn_prefill_workspace_bytes: null output pointer");
  if (n_q_heads < 1 || n_q_heads > 1024 || (head_dim != 64 && head_dim != 128) || m < 1 || m > 65536 || p0 < 0 ||
      p0 + m > kAttnMaxLen)
    return fail(QM_ESHAPE, "qattn_prefill_workspace_bytes: n_q_heads in [1, 1024], head_dim 64 or 128, "
                "1 <= m <= 65536, 0 <= p0, p0 + m <= %lld", (long long)kAttnMaxLen);
  const DeviceInfo* d;
  qm_status st;
  if ((st = device_info(&d)) != QM_OK) return st;
  *bytes = attn_prefill_plan(n_q_heads, head_dim, m, p0, d->cu_count, SIZE_MAX).ws_needed;
  return QM_OK;
}

}  // extern "C"

namespace {

// Shared body of the two prefill-attention entry points (o: fp32 heads, or
// o16: fp16 rows).
qm_status prefill_attention_call(const char* name, const uint16_t* q, const uint16_t* k_cache,
                                 const uint16_t* v_cache, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                 int64_t m, int64_t p0, int64_t max_len, float scale, float* o, uint16_t* o16,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  if (head_dim != 64 && head_dim != 128) return fail(QM_ESHAPE, "%s: head_dim=%d must be 64 or 128", name, head_dim);
  if (n_kv_heads < 1 || n_q_heads < 1 || n_q_heads > 1024 || n_q_heads % n_kv_heads != 0)
    return fail(QM_ESHAPE, "%s: n_q_heads=%d must be a multiple of n_kv_heads=%d", name, n_q_heads, n_kv_heads);
  if (m < 1 || m > 65536 || p0 < 0 || max_len > kAttnMaxLen || p0 + m > max_len)
    return fail(QM_ESHAPE, "%s: need 1 <= m <= 65536, p0 >= 0, p0 + m <= max_len <= %lld", name,
                (long long)kAttnMaxLen);
  if (!(scale > 0.0f) || scale == INFINITY) return fail(QM_EINVAL, "%s: scale must be finite and > 0", name);
  if (!q || !k_cache || !v_cache || (!o && !o16)) return fail(QM_EINVAL, "%s: null pointer", name);
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache))
    return fail(QM_EALIGN, "%s: q, k_cache, v_cache must be 16-byte aligned", name);
  if ((o && !aligned16(o)) || (o16 && !aligned16(o16))) return fail(QM_EALIGN, "%s: the output must be 16-byte aligned", name);
  if (workspace && !aligned16(workspace)) return fail(QM_EALIGN, "%s: workspace must be 16-byte aligned", name);
  const DeviceInfo* d;
  qm_status st;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_attn_prefill(q, k_cache, v_cache, n_q_heads, n_kv_heads, head_dim, m, p0, max_len, scale, o,
                                      o16, workspace, workspace ? workspace_bytes : 0, d->cu_count,
                                      static_cast<hipStream_t>(stream)),
                  name);
}

}  // namespace

extern "C" {

qm_status qattn_prefill(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t n_q_heads,
                        int32_t n_kv_heads, int32_t head_dim, int64_t m, int64_t p0, int64_t max_len, float scale,
                        float* o, void* workspace, size_t workspace_bytes, void* stream) {
  if (!o) return fail(QM_EINVAL, "qattn_prefill: null pointer");
  return prefill_attention_call("qattn_prefill", q, k_cache, v_cache, n_q_heads, n_kv_heads, head_dim, m, p0, max_len,
                                scale, o, nullptr, workspace, workspace_bytes, stream);
}

qm_status qattn_prefill_rows_f16(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                 int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int64_t m, int64_t p0,
                                 int64_t max_len, float scale, uint16_t* out, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  if (!out) return fail(QM_EINVAL, "qattn_prefill_rows_f16: null pointer");
  return prefill_attention_call("qattn_prefill_rows_f16", q, k_cache, v_cache, n_q_heads, n_kv_heads, head_dim, m,
                                p0, max_len, scale, nullptr, out, workspace, workspace_bytes, stream);
}

qm_status qdec_embed(const uint16_t* table, int64_t vocab, int64_t hidden, const int32_t* token, float* x,
                     void* stream) {
  if (vocab < 1 || vocab > INT32_MAX || hidden < 1 || hidden > (int64_t{1} << 20))
    return fail(QM_ESHAPE, "qdec_embed: need 1 <= vocab <= 2^31-1 and 1 <= hidden <= 2^20");
  if (!table || !token || !x) return fail(QM_EINVAL, "qdec_embed: null pointer");
  if (!aligned2(table) || !aligned4(token) || !aligned4(x))
    return fail(QM_EALIGN, "qdec_embed: table 2-byte, token and x 4-byte aligned");
  return launched(launch_embed(table, vocab, hidden, token, x, static_cast<hipStream_t>(stream)), "qdec_embed");
}

qm_status qdec_rmsnorm(float* x, const float* residual, const uint16_t* w, int64_t rows, int64_t hidden, float eps,
                       uint16_t* out, void* stream) {
  if (rows < 0 || rows > 65536 || hidden < 1 || hidden > (int64_t{1} << 20))
    return fail(QM_ESHAPE, "qdec_rmsnorm: need 0 <= rows <= 65536 and 1 <= hidden <= 2^20");
  if (!(eps >= 0.0f) || eps == INFINITY) return fail(QM_EINVAL, "qdec_rmsnorm: eps must be finite and >= 0");
  if (rows > 0 && (!x || !w || !out)) return fail(QM_EINVAL, "qdec_rmsnorm: null pointer");
  if (!aligned4(x) || (residual && !aligned4(residual)) || !aligned2(w) || !aligned2(out))
    return fail(QM_EALIGN, "qdec_rmsnorm: x and residual 4-byte, w and out 2-byte aligned");
  return launched(launch_rmsnorm(x, residual, w, rows, hidden, eps, out, static_cast<hipStream_t>(stream)),
                  "qdec_rmsnorm");
}

qm_status qdec_rope_append(const float* q, const float* k, const float* v, int32_t n_q_heads, int32_t n_kv_heads,
                           int32_t head_dim, int64_t pos, int64_t max_len, float theta, const uint16_t* q_norm,
                           const uint16_t* k_norm, float eps, const float* table, int64_t table_len,
                           uint16_t* q_out, uint16_t* k_cache, uint16_t* v_cache, void* stream) {
  if (table && (!aligned8(table) || table_len <= pos))
    return fail(QM_EINVAL, "qdec_rope_append: the (cos, sin) table must be 8-byte aligned and cover position pos");
  if ((q_norm == nullptr) != (k_norm == nullptr) || !aligned2(q_norm) || !aligned2(k_norm))
    return fail(QM_EINVAL, "qdec_rope_append: q_norm and k_norm both given (2-byte aligned) or both NULL");
  if (q_norm && (!(eps >= 0.0f) || eps == INFINITY)) return fail(QM_EINVAL, "qdec_rope_append: eps finite and >= 0");
  if (head_dim != 64 && head_dim != 128)
    return fail(QM_ESHAPE, "qdec_rope_append: head_dim=%d must be 64 or 128", head_dim);
  if (n_q_heads < 1 || n_q_heads > 1024 || n_kv_heads < 1 || n_kv_heads > 1024)
    return fail(QM_ESHAPE, "qdec_rope_append: head counts must be in [1, 1024]");
  if (max_len < 1 || max_len > kAttnMaxLen || pos < 0 || pos >= max_len)
    return fail(QM_ESHAPE, "qdec_rope_append: need 0 <= pos < max_len <= %lld", (long long)kAttnMaxLen);
  if (!(theta > 1.0f) || theta == INFINITY) return fail(QM_EINVAL, "qdec_rope_append: theta must be finite and > 1");
  if (!q || !k || !v || !q_out || !k_cache || !v_cache) return fail(QM_EINVAL, "qdec_rope_append: null pointer");
  if (!aligned4(q) || !aligned4(k) || !aligned4(v) || !aligned2(q_out) || !aligned2(k_cache) || !aligned2(v_cache))
    return fail(QM_EALIGN, "qdec_rope_append: q, k, v 4-byte, q_out and caches 2-byte aligned");
  return launched(launch_rope_append(q, k, v, n_q_heads, n_kv_heads, head_dim, pos, max_len, theta, q_out, k_cache,
                                     v_cache, q_norm, k_norm, eps, table, static_cast<hipStream_t>(stream)),
                  "qdec_rope_append");
}

qm_status qdec_cast_f16(const float* x, int64_t n, uint16_t* out, void* stream) {
  if (n < 0) return fail(QM_ESHAPE, "qdec_cast_f16: n=%lld must be >= 0", (long long)n);
  if (n > 0 && (!x || !out)) return fail(QM_EINVAL, "qdec_cast_f16: null pointer");
  if (!aligned4(x) || !aligned2(out)) return fail(QM_EALIGN, "qdec_cast_f16: x 4-byte, out 2-byte aligned");
  return launched(launch_cast_f16(x, n, out, static_cast<hipStream_t>(stream)), "qdec_cast_f16");
}

qm_status qdec_argmax(const float* logits, int64_t n, int32_t* token, void* workspace, size_t ws_bytes,
                      void* stream) {
  if (n < 1 || n > INT32_MAX - 1) return fail(QM_ESHAPE, "qdec_argmax: need 1 <= n < 2^31-1");
  if (!logits || !token) return fail(QM_EINVAL, "qdec_argmax: null pointer");
  if (!workspace || ws_bytes < QDEC_ARGMAX_WORKSPACE_BYTES)
    return fail(QM_EWORKSPACE, "qdec_argmax: workspace of %d bytes needed (got %zu)", QDEC_ARGMAX_WORKSPACE_BYTES,
                ws_bytes);
  if (!aligned4(logits) || !aligned4(token) || !aligned4(workspace))
    return fail(QM_EALIGN, "qdec_argmax: logits, token and workspace 4-byte aligned");
  return launched(launch_argmax(logits, n, token, workspace, static_cast<hipStream_t>(stream)), "qdec_argmax");
}

qm_status qmoe_workspace_bytes(int64_t m, int32_t n_experts, int32_t top_k, int64_t hidden, int64_t inter,
                               size_t* bytes) {
  if (!bytes) return fail(QM_EINVAL, "qmoe_workspace_bytes: null output pointer");
  if (m < 0 || m > 65536 || n_experts < 1 || top_k < 1 || top_k > n_experts || top_k > 16 ||
      hidden <= 0 || inter <= 0 || hidden % kGroup || inter % kGroup)
    return fail(QM_ESHAPE, "qmoe_workspace_bytes: bad sizes");
  *bytes = moe_workspace_bytes(m, top_k, hidden, inter);
  return QM_OK;
}

qm_status qmoe_route(const float* logits, int64_t m, int32_t n_experts, int32_t top_k, int32_t* topk_ids,
                     float* topk_w, int32_t* counts, int32_t* offsets, int32_t* sorted_assign,
                     void* stream) {
  if (n_experts < 1 || n_experts > 1024)
    return fail(QM_ESHAPE, "qmoe_route: n_experts=%d must be in [1, 1024]", n_experts);
  if (top_k < 1 || top_k > 16 || top_k > n_experts)
    return fail(QM_ESHAPE, "qmoe_route: top_k=%d must be in [1, min(16, n_experts)]", top_k);
  if (m < 0 || m > 65536) return fail(QM_ESHAPE, "qmoe_route: m=%lld must be in [0, 65536]", (long long)m);
  if (!counts || !offsets) return fail(QM_EINVAL, "qmoe_route: null counts/offsets");
  if (m > 0 && (!logits || !topk_ids || !topk_w || !sorted_assign))
    return fail(QM_EINVAL, "qmoe_route: null pointer");
  if (!aligned4(logits) || !aligned4(topk_ids) || !aligned4(topk_w) || !aligned4(counts) ||
      !aligned4(offsets) || !aligned4(sorted_assign))
    return fail(QM_EALIGN, "qmoe_route: pointers must be 4-byte aligned");
  const DeviceInfo* d;
  qm_status st;
  if ((st = device_info(&d)) != QM_OK) return st;
  return launched(launch_route(logits, m, n_experts, top_k, topk_ids, topk_w, counts, offsets,
                               sorted_assign, static_cast<hipStream_t>(stream)),
                  "qmoe_route");
}

}  // extern "C"

namespace {

// Shared body of the two MoE layer entry points: validation first (nothing
// enqueued on error), then the workspace (the caller's, or the library's
// per-device scratch when noalloc), then the launches.
qm_status moe_layer_call(const char* name, const qm_qweight* w_gate, const qm_qweight* w_up,
                         const qm_qweight* w_down, const uint16_t* x, int64_t m, int32_t top_k,
                         const int32_t* topk_ids, const float* topk_w, const int32_t* counts,
                         const int32_t* offsets, const int32_t* sorted_assign, float* y, void* workspace,
                         size_t ws_bytes, bool noalloc, void* stream) {
  qm_status st;
  if ((st = check_weight(w_gate, name)) != QM_OK) return st;
  if ((st = check_weight(w_up, name)) != QM_OK) return st;
  if ((st = check_weight(w_down, name)) != QM_OK) return st;
  const qm_qweight* ws[3] = {w_gate, w_up, w_down};
  for (const qm_qweight* w : ws) {
    if (w->format != w_gate->format) return fail(QM_EFORMAT, "%s: gate, up and down formats differ", name);
    if (w->format == QM_F16 || w->format == QM_BF16)
      return fail(QM_EFORMAT, "%s: experts must be Q2, Q3, Q4, Q5, Q6 or Q8", name);
    if (w->layout != QM_LAYOUT_DEVICE) return fail(QM_ELAYOUT, "%s: experts must be in DEVICE layout", name);
  }
  const int64_t E = w_gate->batch, inter = w_gate->n, hidden = w_gate->k;
  if (w_up->batch != E || w_up->n != inter || w_up->k != hidden || w_down->batch != E ||
      w_down->n != hidden || w_down->k != inter)
    return fail(QM_ESHAPE, "%s: expert shapes disagree (gate/up [E][inter][hidden], down [E][hidden][inter])",
                name);
  if (E > 1024) return fail(QM_ESHAPE, "%s: at most 1024 experts", name);
  if (inter == 0 || hidden == 0) return fail(QM_ESHAPE, "%s: empty expert matrices", name);
  if (top_k < 1 || top_k > 16 || top_k > E)
    return fail(QM_ESHAPE, "%s: top_k=%d must be in [1, min(16, E)]", name, top_k);
  if (m < 0 || m > 65536) return fail(QM_ESHAPE, "%s: m must be in [0, 65536]", name);
  if (m == 0) return QM_OK;
  if (!x || !topk_ids || !topk_w || !counts || !offsets || !sorted_assign || !y)
    return fail(QM_EINVAL, "%s: null pointer", name);
  if (!aligned16(x) || !aligned16(y)) return fail(QM_EALIGN, "%s: x and y must be 16-byte aligned", name);
  const size_t need = moe_workspace_bytes(m, top_k, hidden, inter);
  if (noalloc) {
    if (need > kMoeScratchBytes)
      return fail(QM_EWORKSPACE, "%s: this layer needs %zu bytes of scratch, more than the %zu the library "
                  "holds per device; use qmoe_grouped_gemm with a workspace or a smaller m", name, need,
                  kMoeScratchBytes);
  } else {
    if (!workspace || ws_bytes < need)
      return fail(QM_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", name, need, ws_bytes);
    if (!aligned16(workspace)) return fail(QM_EALIGN, "%s: workspace must be 16-byte aligned", name);
  }
  const DeviceInfo* d;
  if ((st = device_info(&d)) != QM_OK) return st;
  if (noalloc) {
    const hipError_t e = moe_scratch(&workspace);
    if (e != hipSuccess) return fail(QM_EDEVICE, "%s: scratch lookup failed: %s", name, hipGetErrorString(e));
  }
  MoeArgs a;
  a.gq = static_cast<const uint8_t*>(w_gate->qdata); a.gs = w_gate->scales;
  a.uq = static_cast<const uint8_t*>(w_up->qdata); a.us = w_up->scales;
  a.dq = static_cast<const uint8_t*>(w_down->qdata); a.ds = w_down->scales;
  a.x = x; a.counts = counts; a.offsets = offsets; a.sorted_assign = sorted_assign; a.topk_w = topk_w;
  a.topk_ids = topk_ids;
  a.y = y;
  const size_t h_bytes = (static_cast<size_t>(m * top_k * inter) * 2 + 255) / 256 * 256;
  a.h = static_cast<uint16_t*>(workspace);
  a.yp = reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) + h_bytes);
  a.m = m; a.hidden = hidden; a.inter = inter;
  a.n_experts = static_cast<int32_t>(E); a.top_k = top_k; a.format = w_gate->format;
  return launched(launch_moe(a, d->cu_count, static_cast<hipStream_t>(stream)), name);
}

}  // namespace

extern "C" {

qm_status qmoe_grouped_gemm(const qm_qweight* w_gate, const qm_qweight* w_up, const qm_qweight* w_down,
                            const uint16_t* x, int64_t m, int32_t top_k, const int32_t* topk_ids, const float* topk_w,
                            const int32_t* counts, const int32_t* offsets, const int32_t* sorted_assign, float* y,
                            void* workspace, size_t ws_bytes, void* stream) {
  return moe_layer_call("qmoe_grouped_gemm", w_gate, w_up, w_down, x, m, top_k, topk_ids, topk_w, counts, offsets,
                        sorted_assign, y, workspace, ws_bytes, false, stream);
}

qm_status qmoe_grouped_gemm_noalloc(const qm_qweight* w_gate, const qm_qweight* w_up, const qm_qweight* w_down,
                                    const uint16_t* x, int64_t m, int32_t top_k, const int32_t* topk_ids,
                                    const float* topk_w, const int32_t* counts, const int32_t* offsets,
                                    const int32_t* sorted_assign, float* y, void* stream) {
  return moe_layer_call("qmoe_grouped_gemm_noalloc", w_gate, w_up, w_down, x, m, top_k, topk_ids, topk_w, counts,
                        offsets, sorted_assign, y, nullptr, 0, true, stream);
}

qm_status qm_device_config(char* buf, size_t len) {
  if (!buf || len == 0) return fail(QM_EINVAL, "qm_device_config: null buffer");
  const DeviceInfo* d;
  qm_status st;
  if ((st = device_info(&d)) != QM_OK) return st;
  // The Q4 GEMV kernel of each projection shape of the decode stacks
  // (K -> N), then the prefill and MoE tile choices.
  static const int64_t shapes[][2] = {{1024, 1024}, {1024, 2048}, {2048, 1024}, {1024, 3072}, {3072, 1024},
                                      {1024, 151936}, {3072, 3072}, {3072, 8192}, {8192, 3072},
                                      {3072, 128256}};
  int used = std::snprintf(buf, len, "arch=%s cu=%d", d->arch, d->cu_count);
  for (const auto& sh : shapes) {
    if (used < 0 || static_cast<size_t>(used) >= len) break;
    char name[96];
    gemv_kernel_name(QM_Q4_G32, sh[1], sh[0], d->cu_count, name, sizeof name);
    used += std::snprintf(buf + used, len - used, " gemv_q4(%lld->%lld)=%s", static_cast<long long>(sh[0]),
                          static_cast<long long>(sh[1]), name);
  }
  if (used >= 0 && static_cast<size_t>(used) < len)
    std::snprintf(buf + used, len - used, " gemm_tile(m=512,n=2048)=%s moe_tile(rows/expert=8)=%s "
                  "moe_tile(rows/expert=128)=%s", gemm_tile_name(512, 2048), moe_tile_name(8), moe_tile_name(128));
  return QM_OK;
}

}  // extern "C"
