"""Thin ctypes binding of libqmatmul.so.

Only argument marshalling lives here: torch supplies device memory (for the
outputs it allocates) and the current HIP stream; every step of the
quantised matmul runs in the library's HIP kernels.  The functions carry the
C ABI's names.  If the library has not been built, every call raises: there
is no fallback path.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

Q4_G32, Q8_G32, Q2_G32, Q3_G32, Q5_G32, Q6_G32, F16, BF16 = 1, 2, 3, 4, 5, 6, 7, 8
LAYOUT_CANONICAL, LAYOUT_DEVICE = 0, 1

STATUS = {0: "QM_OK", 1: "QM_EINVAL", 2: "QM_ESHAPE", 3: "QM_EALIGN", 4: "QM_EFORMAT",
          5: "QM_ELAYOUT", 6: "QM_EWORKSPACE", 7: "QM_EDEVICE"}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libqmatmul.so")

EXPORTS = ("qm_last_error", "qm_weight_bytes", "qm_quantise", "qm_dequantise", "qm_repack",
           "qmatmul_gemv", "qmatmul_gemv_swiglu", "qmatmul_gemv_grouped", "qmatmul_gemm",
           "qmatmul_gemm_grouped",
           "qmoe_workspace_bytes", "qmoe_route",
           "qmoe_grouped_gemm", "qmoe_grouped_gemm_noalloc", "qm_device_config", "qattn_decode_workspace_bytes", "qattn_decode",
           "qattn_prefill", "qdec_embed", "qdec_rmsnorm", "qdec_rope_append", "qdec_cast_f16",
           "qdec_argmax", "qmatmul_gemv_swiglu_f16", "qattn_decode_f16", "qmatmul_gemv_grouped_rmsnorm",
           "qmatmul_gemv_swiglu_rmsnorm_f16", "qdec_rope_table", "qdec_rope_table_llama3",
           "qmatmul_gemv_qkv_rmsnorm_rope", "qdec_embed_rows", "qdec_rope_append_rows", "qdec_heads_to_rows_f16",
           "qdec_swiglu_f16", "qattn_prefill_workspace_bytes", "qattn_prefill_rows_f16")


class QmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class CQWeight(ctypes.Structure):
    _fields_ = [("format", ctypes.c_int32), ("layout", ctypes.c_int32), ("batch", ctypes.c_int64),
                ("n", ctypes.c_int64), ("k", ctypes.c_int64), ("qdata", ctypes.c_void_p),
                ("scales", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    """Loads libqmatmul.so (raises if it was never built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2607_00501_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        W = ctypes.POINTER(CQWeight)
        L.qm_last_error.restype = ctypes.c_char_p
        L.qm_last_error.argtypes = []
        sig = {
            "qm_weight_bytes": [i32, i32, i64, i64, i64, ctypes.POINTER(sz), ctypes.POINTER(sz)],
            "qm_quantise": [i32, vp, W, vp],
            "qm_dequantise": [W, vp, vp],
            "qm_repack": [W, W, vp],
            "qmatmul_gemv": [W, vp, vp, vp],
            "qmatmul_gemv_swiglu": [W, W, vp, vp, vp],
            "qmatmul_gemv_grouped": [i32, W, ctypes.POINTER(vp), ctypes.POINTER(vp), vp],
            "qmatmul_gemm": [W, vp, i64, vp, vp],
            "qmatmul_gemm_grouped": [i32, W, vp, i64, ctypes.POINTER(vp), vp],
            "qmoe_workspace_bytes": [i64, i32, i32, i64, i64, ctypes.POINTER(sz)],
            "qmoe_route": [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp],
            "qmoe_grouped_gemm": [W, W, W, vp, i64, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp],
            "qmoe_grouped_gemm_noalloc": [W, W, W, vp, i64, i32, vp, vp, vp, vp, vp, vp, vp],
            "qm_device_config": [ctypes.c_char_p, sz],
            "qattn_decode_workspace_bytes": [i32, i32, ctypes.POINTER(sz)],
            "qattn_decode": [vp, vp, vp, i32, i32, i32, i64, i64, ctypes.c_float, vp, vp, sz, vp],
            "qattn_prefill": [vp, vp, vp, i32, i32, i32, i64, i64, i64, ctypes.c_float, vp, vp, sz, vp],
            "qattn_prefill_workspace_bytes": [i32, i32, i64, i64, ctypes.POINTER(sz)],
            "qattn_prefill_rows_f16": [vp, vp, vp, i32, i32, i32, i64, i64, i64, ctypes.c_float, vp, vp, sz, vp],
            "qdec_embed": [vp, i64, i64, vp, vp, vp],
            "qmatmul_gemv_swiglu_f16": [W, W, vp, vp, vp],
            "qdec_rope_table": [i64, i32, ctypes.c_float, vp, vp],
            "qdec_rope_table_llama3": [i64, i32, ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                       ctypes.c_float, vp, vp],
            "qdec_embed_rows": [vp, i64, i64, vp, i64, vp, vp],
            "qdec_rope_append_rows": [vp, vp, vp, i32, i32, i32, i64, i64, i64, ctypes.c_float, i32, vp, vp,
                                      ctypes.c_float, vp, i64, vp, vp, vp, vp],
            "qdec_heads_to_rows_f16": [vp, i32, i64, i32, vp, vp],
            "qdec_swiglu_f16": [vp, vp, i64, vp, vp],
            "qmatmul_gemv_qkv_rmsnorm_rope": [W, vp, vp, vp, ctypes.c_float, vp, i32, i32, i32, i64, i64, vp, vp, vp,
                                              vp, vp],
            "qmatmul_gemv_grouped_rmsnorm": [i32, W, vp, vp, vp, ctypes.c_float, vp, ctypes.POINTER(vp), vp],
            "qmatmul_gemv_swiglu_rmsnorm_f16": [W, W, vp, vp, vp, ctypes.c_float, vp, vp, vp],
            "qattn_decode_f16": [vp, vp, vp, i32, i32, i32, i64, i64, ctypes.c_float, vp, vp, sz, vp],
            "qdec_rmsnorm": [vp, vp, vp, i64, i64, ctypes.c_float, vp, vp],
            "qdec_rope_append": [vp, vp, vp, i32, i32, i32, i64, i64, ctypes.c_float, vp, vp, ctypes.c_float, vp, i64,
                                 vp, vp, vp, vp],
            "qdec_cast_f16": [vp, i64, vp, vp],
            "qdec_argmax": [vp, i64, vp, vp, sz, vp],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != 0:
        raise QmError(status, lib().qm_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


@dataclass
class QWeight:
    """A quantised tensor [batch][n][k]: codes and fp16 scale bits in torch
    uint8 / int16 buffers, in CANONICAL or DEVICE layout (F16/BF16: the
    uint16 patterns as bytes; the scale buffer is a 1-element placeholder)."""
    format: int
    layout: int
    batch: int
    n: int
    k: int
    qdata: torch.Tensor
    scales: torch.Tensor

    def c(self) -> CQWeight:
        return CQWeight(self.format, self.layout, self.batch, self.n, self.k,
                        self.qdata.data_ptr(), self.scales.data_ptr())

    @property
    def nbytes(self) -> int:
        return self.qdata.numel() + 2 * self.scales.numel()


def qm_last_error() -> str:
    return lib().qm_last_error().decode()


def qm_weight_bytes(fmt: int, layout: int, batch: int, n: int, k: int):
    qb, sb = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().qm_weight_bytes(fmt, layout, batch, n, k, ctypes.byref(qb), ctypes.byref(sb)))
    return qb.value, sb.value


def empty_qweight(fmt: int, layout: int, batch: int, n: int, k: int, device="cuda") -> QWeight:
    qb, sb = qm_weight_bytes(fmt, layout, batch, n, k)
    return QWeight(fmt, layout, batch, n, k,
                   torch.empty(max(qb, 1), dtype=torch.uint8, device=device),
                   torch.empty(max(sb // 2, 1), dtype=torch.int16, device=device))


def qm_quantise(w: torch.Tensor, fmt: int, out: Optional[QWeight] = None, stream=None) -> QWeight:
    """w: fp32 [n][k] or [batch][n][k] on the GPU -> CANONICAL QWeight."""
    if w.dim() == 2:
        batch, (n, k) = 1, w.shape
    else:
        batch, n, k = w.shape
    assert w.dtype == torch.float32 and w.is_contiguous()
    if out is None:
        out = empty_qweight(fmt, LAYOUT_CANONICAL, batch, n, k, w.device)
    _check(lib().qm_quantise(fmt, _ptr(w), ctypes.byref(out.c()), _stream(stream)))
    return out


def qm_dequantise(w: QWeight, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    if out is None:
        out = torch.empty((w.batch, w.n, w.k), dtype=torch.float32, device=w.qdata.device)
    _check(lib().qm_dequantise(ctypes.byref(w.c()), _ptr(out), _stream(stream)))
    return out


def qm_repack(src: QWeight, layout: int, out: Optional[QWeight] = None, stream=None) -> QWeight:
    if out is None:
        out = empty_qweight(src.format, layout, src.batch, src.n, src.k, src.qdata.device)
    _check(lib().qm_repack(ctypes.byref(src.c()), ctypes.byref(out.c()), _stream(stream)))
    return out


def qmatmul_gemv(w: QWeight, x: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """x: fp16 [k] -> fp32 [n]."""
    assert x.dtype == torch.float16 and x.is_contiguous() and x.numel() == w.k
    if out is None:
        out = torch.empty(w.n, dtype=torch.float32, device=x.device)
    _check(lib().qmatmul_gemv(ctypes.byref(w.c()), _ptr(x), _ptr(out), _stream(stream)))
    return out


def qmatmul_gemv_swiglu(w_gate: QWeight, w_up: QWeight, x: torch.Tensor, out: Optional[torch.Tensor] = None,
                        stream=None):
    """x: fp16 [k] -> h = silu(Wg x) * (Wu x), fp32 [n] (fp16 when `out` is
    an fp16 tensor)."""
    assert x.dtype == torch.float16 and x.is_contiguous() and x.numel() == w_gate.k
    if out is None:
        out = torch.empty(w_gate.n, dtype=torch.float32, device=x.device)
    fn = lib().qmatmul_gemv_swiglu_f16 if out.dtype == torch.float16 else lib().qmatmul_gemv_swiglu
    assert out.dtype in (torch.float16, torch.float32) and out.is_contiguous() and out.numel() == w_gate.n
    _check(fn(ctypes.byref(w_gate.c()), ctypes.byref(w_up.c()), _ptr(x), _ptr(out), _stream(stream)))
    return out


GEMV_GROUP_MAX = 8


def gemv_group_args(ws, xs, outs):
    """Marshals a grouped GEMV call: (count, descriptor array, x pointer
    array, y pointer array); keep the returned tuple alive while in use."""
    n = len(ws)
    descs = (CQWeight * n)(*[w.c() for w in ws])
    xp = (ctypes.c_void_p * n)(*[t.data_ptr() for t in xs])
    yp = (ctypes.c_void_p * n)(*[t.data_ptr() for t in outs])
    return n, descs, xp, yp


def qmatmul_gemv_grouped(ws, xs, outs=None, stream=None):
    """Independent GEMVs y_i = W_i' x_i with one k, in one launch; xs may repeat
    a tensor (shared input).  Returns the list of fp32 outputs."""
    assert len(ws) == len(xs)
    for w, x in zip(ws, xs):
        assert x.dtype == torch.float16 and x.is_contiguous() and x.numel() == w.k
    if outs is None:
        outs = [torch.empty(w.n, dtype=torch.float32, device=x.device) for w, x in zip(ws, xs)]
    n, descs, xp, yp = gemv_group_args(ws, xs, outs)
    _check(lib().qmatmul_gemv_grouped(n, descs, xp, yp, _stream(stream)))
    return outs


def qmatmul_gemv_grouped_rmsnorm(ws, x: torch.Tensor, gain: torch.Tensor, eps: float, x_out: torch.Tensor,
                                 residual: Optional[torch.Tensor] = None, outs=None, stream=None):
    """y_i = W_i' fp16(rmsnorm(x + residual) * gain); x_out = x + residual
    (fp32 [k]).  Returns the list of fp32 outputs."""
    k = ws[0].k
    for t in (x, x_out) + ((residual,) if residual is not None else ()):
        assert t.dtype == torch.float32 and t.is_contiguous() and t.numel() == k
    assert gain.dtype == torch.float16 and gain.numel() == k
    if outs is None:
        outs = [torch.empty(w.n, dtype=torch.float32, device=x.device) for w in ws]
    n = len(ws)
    descs = (CQWeight * n)(*[w.c() for w in ws])
    yp = (ctypes.c_void_p * n)(*[t.data_ptr() for t in outs])
    _check(lib().qmatmul_gemv_grouped_rmsnorm(n, descs, _ptr(x), _ptr(residual), _ptr(gain), eps, _ptr(x_out), yp,
                                              _stream(stream)))
    return outs


def qmatmul_gemv_swiglu_rmsnorm_f16(w_gate: QWeight, w_up: QWeight, x: torch.Tensor, gain: torch.Tensor, eps: float,
                                    x_out: torch.Tensor, residual: Optional[torch.Tensor] = None,
                                    out: Optional[torch.Tensor] = None, stream=None):
    """h = fp16(silu(Wg' n) * (Wu' n)), n = fp16(rmsnorm(x + residual) * gain);
    x_out = x + residual."""
    k = w_gate.k
    for t in (x, x_out) + ((residual,) if residual is not None else ()):
        assert t.dtype == torch.float32 and t.is_contiguous() and t.numel() == k
    assert gain.dtype == torch.float16 and gain.numel() == k
    if out is None:
        out = torch.empty(w_gate.n, dtype=torch.float16, device=x.device)
    assert out.dtype == torch.float16 and out.numel() == w_gate.n
    _check(lib().qmatmul_gemv_swiglu_rmsnorm_f16(ctypes.byref(w_gate.c()), ctypes.byref(w_up.c()), _ptr(x),
                                                 _ptr(residual), _ptr(gain), eps, _ptr(x_out), _ptr(out),
                                                 _stream(stream)))
    return out


def qdec_embed_rows(table: torch.Tensor, tokens: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """table fp16 [vocab][hidden], tokens int32 [m] (device) -> fp32 [m][hidden]."""
    vocab, hidden = table.shape
    m = tokens.numel()
    assert tokens.dtype == torch.int32 and table.dtype == torch.float16
    if out is None:
        out = torch.empty((m, hidden), dtype=torch.float32, device=table.device)
    _check(lib().qdec_embed_rows(_ptr(table), vocab, hidden, _ptr(tokens), m, _ptr(out), _stream(stream)))
    return out


def _check_head_gains(q_norm, k_norm, d):
    """The per-head q/k norm gains: both absent, or fp16 contiguous [D] each
    (the kernel reads exactly D fp16 values from each pointer)."""
    assert (q_norm is None) == (k_norm is None), "q_norm and k_norm go together"
    for g in (q_norm, k_norm):
        if g is not None:
            assert g.dtype == torch.float16 and g.is_contiguous() and g.numel() == d, \
                "q/k norm gains must be fp16, contiguous, head_dim elements"


def qdec_rope_append_rows(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, p0: int, theta: float,
                          k_cache: torch.Tensor, v_cache: torch.Tensor, interleaved: bool = False,
                          q_out: Optional[torch.Tensor] = None, q_norm: Optional[torch.Tensor] = None,
                          k_norm: Optional[torch.Tensor] = None, eps: float = 1e-6,
                          table: Optional[torch.Tensor] = None, stream=None):
    """q fp32 [m][Hq*D], k, v fp32 [m][Hkv*D] -> fp16 [Hq][m][D]; cache rows p0..p0+m-1.
    table: qdec_rope_table's [positions][D/2][2] fp32 for this theta and D
    (read instead of computing each angle)."""
    hkv, max_len, d = k_cache.shape
    m = q.shape[0]
    hq = q.shape[1] // d
    assert q.dtype == k.dtype == v.dtype == torch.float32 and k.shape == v.shape == (m, hkv * d)
    assert q.is_contiguous() and k.is_contiguous() and v.is_contiguous() and q.shape[1] == hq * d
    assert k_cache.dtype == v_cache.dtype == torch.float16 and v_cache.shape == k_cache.shape
    assert k_cache.is_contiguous() and v_cache.is_contiguous()
    _check_head_gains(q_norm, k_norm, d)
    if q_out is None:
        q_out = torch.empty((hq, m, d), dtype=torch.float16, device=q.device)
    tlen = 0
    if table is not None:
        assert table.dtype == torch.float32 and table.is_contiguous() and table.shape[1:] == (d // 2, 2)
        tlen = table.shape[0]
    _check(lib().qdec_rope_append_rows(_ptr(q), _ptr(k), _ptr(v), hq, hkv, d, m, p0, max_len, theta,
                                       1 if interleaved else 0, _ptr(q_norm), _ptr(k_norm), eps, _ptr(table), tlen,
                                       _ptr(q_out), _ptr(k_cache), _ptr(v_cache), _stream(stream)))
    return q_out


def qdec_heads_to_rows_f16(o: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """fp32 [H][m][D] -> fp16 [m][H*D]."""
    h, m, d = o.shape
    if out is None:
        out = torch.empty((m, h * d), dtype=torch.float16, device=o.device)
    _check(lib().qdec_heads_to_rows_f16(_ptr(o), h, m, d, _ptr(out), _stream(stream)))
    return out


def qdec_swiglu_f16(gate: torch.Tensor, up: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """fp16(silu(gate) * up), elementwise, fp32 in."""
    assert gate.dtype == up.dtype == torch.float32 and gate.shape == up.shape
    if out is None:
        out = torch.empty(gate.shape, dtype=torch.float16, device=gate.device)
    _check(lib().qdec_swiglu_f16(_ptr(gate), _ptr(up), gate.numel(), _ptr(out), _stream(stream)))
    return out


def qdec_rope_table(max_len: int, head_dim: int, theta: float, device="cuda", stream=None) -> torch.Tensor:
    """fp32 [max_len][head_dim/2][2] (cos, sin) table."""
    t = torch.empty((max_len, head_dim // 2, 2), dtype=torch.float32, device=device)
    _check(lib().qdec_rope_table(max_len, head_dim, theta, _ptr(t), _stream(stream)))
    return t


def qdec_rope_table_llama3(max_len: int, head_dim: int, theta: float, scaling, device="cuda",
                           stream=None) -> torch.Tensor:
    """The (cos, sin) table with the Llama 3 long-context frequencies;
    scaling = (factor, low_freq_factor, high_freq_factor, original_len)."""
    factor, low, high, orig = (float(v) for v in scaling)
    t = torch.empty((max_len, head_dim // 2, 2), dtype=torch.float32, device=device)
    _check(lib().qdec_rope_table_llama3(max_len, head_dim, theta, factor, low, high, orig, _ptr(t), _stream(stream)))
    return t


def rope_interleave_rows(w: torch.Tensor, n_heads: int, head_dim: int) -> torch.Tensor:
    """Row order qmatmul_gemv_qkv_rmsnorm_rope expects for W_q / W_k: within
    each head, stored row 2i = row i and stored row 2i + 1 = row i + D/2."""
    k = w.shape[-1]
    return w.reshape(n_heads, 2, head_dim // 2, k).transpose(1, 2).reshape(n_heads * head_dim, k).contiguous()


def qmatmul_gemv_qkv_rmsnorm_rope(ws, x: torch.Tensor, gain: torch.Tensor, eps: float, x_out: torch.Tensor,
                                  pos: int, rope_table: torch.Tensor, q_out: torch.Tensor, k_cache: torch.Tensor,
                                  v_cache: torch.Tensor, residual: Optional[torch.Tensor] = None, stream=None):
    """q/k/v GEMV with the norm folded in and RoPE + cache append as the
    epilogue (ws[0], ws[1] with rope_interleave_rows order)."""
    hkv, max_len, d = k_cache.shape
    hq = ws[0].n // d
    k = ws[0].k
    for t in (x, x_out) + ((residual,) if residual is not None else ()):
        assert t.dtype == torch.float32 and t.is_contiguous() and t.numel() == k
    assert gain.dtype == torch.float16 and gain.numel() == k
    assert q_out.dtype == k_cache.dtype == v_cache.dtype == torch.float16 and q_out.numel() == hq * d
    assert rope_table.dtype == torch.float32 and rope_table.shape == (max_len, d // 2, 2)
    descs = (CQWeight * 3)(*[w.c() for w in ws])
    _check(lib().qmatmul_gemv_qkv_rmsnorm_rope(descs, _ptr(x), _ptr(residual), _ptr(gain), eps, _ptr(x_out), hq,
                                               hkv, d, pos, max_len, _ptr(rope_table), _ptr(q_out),
                                               _ptr(k_cache), _ptr(v_cache), _stream(stream)))
    return q_out


def qmatmul_gemm(w: QWeight, x: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """X: fp16 [m][k] -> fp32 [m][n]."""
    assert x.dtype == torch.float16 and x.is_contiguous() and x.dim() == 2 and x.shape[1] == w.k
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, w.n), dtype=torch.float32, device=x.device)
    _check(lib().qmatmul_gemm(ctypes.byref(w.c()), _ptr(x), m, _ptr(out), _stream(stream)))
    return out


def gemm_group_args(ws, outs):
    """Marshals a grouped GEMM call: (count, descriptor array, y pointer
    array); keep the returned tuple alive while in use."""
    n = len(ws)
    descs = (CQWeight * n)(*[w.c() for w in ws])
    yp = (ctypes.c_void_p * n)(*[t.data_ptr() for t in outs])
    return n, descs, yp


def qmatmul_gemm_grouped(ws, x: torch.Tensor, outs=None, stream=None):
    """Y_i = X W_i'^T for matrices with one k sharing X, in one launch."""
    assert x.dtype == torch.float16 and x.is_contiguous() and x.dim() == 2
    m = x.shape[0]
    for w in ws:
        assert x.shape[1] == w.k
    if outs is None:
        outs = [torch.empty((m, w.n), dtype=torch.float32, device=x.device) for w in ws]
    n, descs, yp = gemm_group_args(ws, outs)
    _check(lib().qmatmul_gemm_grouped(n, descs, _ptr(x), m, yp, _stream(stream)))
    return outs


def qattn_decode_workspace_bytes(n_q_heads: int, head_dim: int) -> int:
    b = ctypes.c_size_t()
    _check(lib().qattn_decode_workspace_bytes(n_q_heads, head_dim, ctypes.byref(b)))
    return b.value


def qattn_decode(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, length: int, scale: float,
                 out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None, stream=None):
    """q: fp16 [Hq][D]; k_cache, v_cache: fp16 [Hkv][max_len][D] -> fp32 [Hq][D]
    (fp16 when `out` is an fp16 tensor)."""
    hq, d = q.shape
    hkv, max_len, d2 = k_cache.shape
    assert d2 == d and v_cache.shape == k_cache.shape
    assert q.dtype == k_cache.dtype == v_cache.dtype == torch.float16
    assert q.is_contiguous() and k_cache.is_contiguous() and v_cache.is_contiguous()
    if out is None:
        out = torch.empty((hq, d), dtype=torch.float32, device=q.device)
    nb = qattn_decode_workspace_bytes(hq, d)
    if workspace is None:
        workspace = torch.empty(nb, dtype=torch.uint8, device=q.device)
    assert out.dtype in (torch.float16, torch.float32) and out.is_contiguous() and out.numel() == hq * d
    fn = lib().qattn_decode_f16 if out.dtype == torch.float16 else lib().qattn_decode
    _check(fn(_ptr(q), _ptr(k_cache), _ptr(v_cache), hq, hkv, d, length, max_len, scale,
              _ptr(out), _ptr(workspace), workspace.numel(), _stream(stream)))
    return out


def qattn_prefill_workspace_bytes(n_q_heads: int, head_dim: int, m: int, p0: int) -> int:
    b = ctypes.c_size_t()
    _check(lib().qattn_prefill_workspace_bytes(n_q_heads, head_dim, m, p0, ctypes.byref(b)))
    return b.value


NO_WORKSPACE = object()   # qattn_prefill without a workspace (no key splits)


def qattn_prefill(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, p0: int, scale: float,
                  out: Optional[torch.Tensor] = None, workspace=None, stream=None):
    """q: fp16 [Hq][m][D] at positions p0..p0+m-1; k_cache, v_cache: fp16
    [Hkv][max_len][D] -> fp32 [Hq][m][D] (causal).  workspace: a uint8
    device tensor for the key-split partials (allocated at the full plan's
    size when None; pass binding.NO_WORKSPACE for the single-launch,
    unsplit form)."""
    hq, m, d = q.shape
    hkv, max_len, d2 = k_cache.shape
    assert d2 == d and v_cache.shape == k_cache.shape
    assert q.dtype == k_cache.dtype == v_cache.dtype == torch.float16
    assert q.is_contiguous() and k_cache.is_contiguous() and v_cache.is_contiguous()
    if out is None:
        out = torch.empty((hq, m, d), dtype=torch.float32, device=q.device)
    assert out.dtype == torch.float32 and out.is_contiguous() and out.numel() == hq * m * d
    if workspace is None:
        nb = qattn_prefill_workspace_bytes(hq, d, m, p0)
        workspace = torch.empty(max(nb, 16), dtype=torch.uint8, device=q.device)
    if workspace is NO_WORKSPACE:
        wp, wn = None, 0
    else:
        assert workspace.dtype == torch.uint8 and workspace.is_contiguous()
        wp, wn = _ptr(workspace), workspace.numel()
    _check(lib().qattn_prefill(_ptr(q), _ptr(k_cache), _ptr(v_cache), hq, hkv, d, m, p0, max_len, scale,
                               _ptr(out), wp, wn, _stream(stream)))
    return out


def qattn_prefill_rows_f16(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, p0: int, scale: float,
                           out: Optional[torch.Tensor] = None, workspace=None, stream=None):
    """qattn_prefill with fp16 rows out: [m][Hq * D] (the o-projection GEMM's
    input).  workspace as for qattn_prefill."""
    hq, m, d = q.shape
    hkv, max_len, d2 = k_cache.shape
    assert d2 == d and v_cache.shape == k_cache.shape
    assert q.dtype == k_cache.dtype == v_cache.dtype == torch.float16
    assert q.is_contiguous() and k_cache.is_contiguous() and v_cache.is_contiguous()
    if out is None:
        out = torch.empty((m, hq * d), dtype=torch.float16, device=q.device)
    assert out.dtype == torch.float16 and out.is_contiguous() and out.numel() == hq * m * d
    if workspace is None:
        nb = qattn_prefill_workspace_bytes(hq, d, m, p0)
        workspace = torch.empty(max(nb, 16), dtype=torch.uint8, device=q.device)
    if workspace is NO_WORKSPACE:
        wp, wn = None, 0
    else:
        assert workspace.dtype == torch.uint8 and workspace.is_contiguous()
        wp, wn = _ptr(workspace), workspace.numel()
    _check(lib().qattn_prefill_rows_f16(_ptr(q), _ptr(k_cache), _ptr(v_cache), hq, hkv, d, m, p0, max_len, scale,
                                        _ptr(out), wp, wn, _stream(stream)))
    return out


def qdec_embed(table: torch.Tensor, token: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """table: fp16 [vocab][hidden]; token: int32 [1] on the device -> fp32 [hidden]."""
    vocab, hidden = table.shape
    assert table.dtype == torch.float16 and table.is_contiguous() and token.dtype == torch.int32
    if out is None:
        out = torch.empty(hidden, dtype=torch.float32, device=table.device)
    _check(lib().qdec_embed(_ptr(table), vocab, hidden, _ptr(token), _ptr(out), _stream(stream)))
    return out


def qdec_rmsnorm(x: torch.Tensor, w: torch.Tensor, eps: float, residual: Optional[torch.Tensor] = None,
                 out: Optional[torch.Tensor] = None, stream=None):
    """x: fp32 [rows][hidden] or [hidden] (updated in place when residual is
    given: x += residual); w: fp16 [hidden] -> fp16 like x."""
    hidden = x.shape[-1]
    rows = x.numel() // hidden if hidden else 0
    assert x.dtype == torch.float32 and x.is_contiguous() and w.dtype == torch.float16 and w.numel() == hidden
    if residual is not None:
        assert residual.dtype == torch.float32 and residual.shape == x.shape and residual.is_contiguous()
    if out is None:
        out = torch.empty(x.shape, dtype=torch.float16, device=x.device)
    _check(lib().qdec_rmsnorm(_ptr(x), _ptr(residual), _ptr(w), rows, hidden, eps, _ptr(out), _stream(stream)))
    return out


def qdec_rope_append(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, pos: int, theta: float,
                     k_cache: torch.Tensor, v_cache: torch.Tensor, q_out: Optional[torch.Tensor] = None,
                     q_norm: Optional[torch.Tensor] = None, k_norm: Optional[torch.Tensor] = None, eps: float = 1e-6,
                     table: Optional[torch.Tensor] = None, stream=None):
    """q: fp32 [Hq*D]; k, v: fp32 [Hkv*D]; caches fp16 [Hkv][max_len][D]
    (row pos written) -> fp16 [Hq][D] rotated queries.  table: qdec_rope_table's
    (cos, sin) for this theta and D, read instead of computing the angles."""
    hkv, max_len, d = k_cache.shape
    hq = q.numel() // d
    assert q.dtype == k.dtype == v.dtype == torch.float32 and k.numel() == v.numel() == hkv * d
    assert k_cache.dtype == v_cache.dtype == torch.float16 and v_cache.shape == k_cache.shape
    assert k_cache.is_contiguous() and v_cache.is_contiguous()
    _check_head_gains(q_norm, k_norm, d)
    if q_out is None:
        q_out = torch.empty((hq, d), dtype=torch.float16, device=q.device)
    tlen = 0
    if table is not None:
        assert table.dtype == torch.float32 and table.is_contiguous() and table.shape[1:] == (d // 2, 2)
        tlen = table.shape[0]
    _check(lib().qdec_rope_append(_ptr(q), _ptr(k), _ptr(v), hq, hkv, d, pos, max_len, theta, _ptr(q_norm),
                                  _ptr(k_norm), eps, _ptr(table), tlen, _ptr(q_out), _ptr(k_cache), _ptr(v_cache),
                                  _stream(stream)))
    return q_out


def qdec_cast_f16(x: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """fp32 -> fp16 (round to nearest even), any shape."""
    assert x.dtype == torch.float32 and x.is_contiguous()
    if out is None:
        out = torch.empty(x.shape, dtype=torch.float16, device=x.device)
    _check(lib().qdec_cast_f16(_ptr(x), x.numel(), _ptr(out), _stream(stream)))
    return out


ARGMAX_WORKSPACE_BYTES = 2048


def qdec_argmax(logits: torch.Tensor, out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                stream=None):
    """fp32 [n] -> int32 [1] on the device (lowest index among equal maxima)."""
    assert logits.dtype == torch.float32 and logits.is_contiguous()
    if out is None:
        out = torch.empty(1, dtype=torch.int32, device=logits.device)
    if workspace is None:
        workspace = torch.empty(ARGMAX_WORKSPACE_BYTES, dtype=torch.uint8, device=logits.device)
    _check(lib().qdec_argmax(_ptr(logits), logits.numel(), _ptr(out), _ptr(workspace), workspace.numel(),
                             _stream(stream)))
    return out


def qmoe_workspace_bytes(m: int, n_experts: int, top_k: int, hidden: int, inter: int) -> int:
    b = ctypes.c_size_t()
    _check(lib().qmoe_workspace_bytes(m, n_experts, top_k, hidden, inter, ctypes.byref(b)))
    return b.value


@dataclass
class Routing:
    ids: torch.Tensor            # int32 [m][top_k]
    gates: torch.Tensor          # fp32 [m][top_k]
    counts: torch.Tensor         # int32 [E]
    offsets: torch.Tensor        # int32 [E+1]
    sorted_assign: torch.Tensor  # int32 [m*top_k]
    top_k: int


def qmoe_route(logits: torch.Tensor, top_k: int, out: Optional[Routing] = None, stream=None) -> Routing:
    m, e = logits.shape
    assert logits.dtype == torch.float32 and logits.is_contiguous()
    dev = logits.device
    if out is None:
        out = Routing(torch.empty((m, top_k), dtype=torch.int32, device=dev),
                      torch.empty((m, top_k), dtype=torch.float32, device=dev),
                      torch.empty(e, dtype=torch.int32, device=dev),
                      torch.empty(e + 1, dtype=torch.int32, device=dev),
                      torch.empty(max(m * top_k, 1), dtype=torch.int32, device=dev), top_k)
    _check(lib().qmoe_route(_ptr(logits), m, e, top_k, _ptr(out.ids), _ptr(out.gates), _ptr(out.counts),
                            _ptr(out.offsets), _ptr(out.sorted_assign), _stream(stream)))
    return out


def qmoe_grouped_gemm(w_gate: QWeight, w_up: QWeight, w_down: QWeight, x: torch.Tensor, r: Routing,
                      out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    m, hidden = x.shape
    assert x.dtype == torch.float16 and x.is_contiguous()
    if out is None:
        out = torch.empty((m, hidden), dtype=torch.float32, device=x.device)
    if workspace is None:
        nb = qmoe_workspace_bytes(m, w_gate.batch, r.top_k, hidden, w_gate.n)
        workspace = torch.empty(max(nb, 16), dtype=torch.uint8, device=x.device)
    _check(lib().qmoe_grouped_gemm(ctypes.byref(w_gate.c()), ctypes.byref(w_up.c()), ctypes.byref(w_down.c()),
                                   _ptr(x), m, r.top_k, _ptr(r.ids), _ptr(r.gates), _ptr(r.counts), _ptr(r.offsets),
                                   _ptr(r.sorted_assign), _ptr(out), _ptr(workspace), workspace.numel(),
                                   _stream(stream)))
    return out


NOALLOC_SCRATCH_BYTES = 32 << 20     # QMOE_NOALLOC_SCRATCH_BYTES


def qmoe_grouped_gemm_noalloc(w_gate: QWeight, w_up: QWeight, w_down: QWeight, x: torch.Tensor, r: Routing,
                              out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """qmoe_grouped_gemm with the library's per-device scratch instead of a
    caller workspace (the C call allocates nothing; `out` is allocated here
    only when not given)."""
    m, hidden = x.shape
    assert x.dtype == torch.float16 and x.is_contiguous()
    if out is None:
        out = torch.empty((m, hidden), dtype=torch.float32, device=x.device)
    _check(lib().qmoe_grouped_gemm_noalloc(ctypes.byref(w_gate.c()), ctypes.byref(w_up.c()),
                                           ctypes.byref(w_down.c()), _ptr(x), m, r.top_k, _ptr(r.ids),
                                           _ptr(r.gates), _ptr(r.counts), _ptr(r.offsets), _ptr(r.sorted_assign),
                                           _ptr(out), _stream(stream)))
    return out


def qm_device_config() -> str:
    buf = ctypes.create_string_buffer(4096)
    _check(lib().qm_device_config(buf, 4096))
    return buf.value.decode()
