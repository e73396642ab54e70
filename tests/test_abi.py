"""Host-side checks of the C ABI (no GPU needed): the library loads and
exports every function include/qmatmul.h declares, the pure host functions
return the documented sizes, and invalid arguments are rejected before any
device work with the documented status and a message."""

import ctypes
import os
import re

import pytest

from paper_2607_00501_amd import binding as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "qmatmul.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(q\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    names = _declared_functions()
    assert len(names) >= 11, names
    lib = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.EXPORTS)


@pytest.mark.parametrize("fmt,layout,batch,n,k,want", [
    (B.Q4_G32, B.LAYOUT_CANONICAL, 1, 3, 64, (3 * 32, 3 * 2 * 2)),
    (B.Q4_G32, B.LAYOUT_DEVICE, 1, 3, 64, (64 * 32, 64 * 2 * 2)),
    (B.Q8_G32, B.LAYOUT_DEVICE, 2, 65, 32, (2 * 128 * 32, 2 * 128 * 2)),
    (B.Q4_G32, B.LAYOUT_DEVICE, 1, 151936, 1024, (151936 * 512, 151936 * 32 * 2)),
    (B.Q8_G32, B.LAYOUT_CANONICAL, 128, 768, 2048, (128 * 768 * 2048, 128 * 768 * 64 * 2)),
    (B.Q2_G32, B.LAYOUT_DEVICE, 1, 3, 64, (64 * 64 * 2 // 8, 64 * 2 * 2)),
    (B.Q3_G32, B.LAYOUT_CANONICAL, 2, 5, 96, (2 * 5 * 96 * 3 // 8, 2 * 5 * 3 * 2)),
    (B.Q5_G32, B.LAYOUT_DEVICE, 1, 65, 32, (128 * 32 * 5 // 8, 128 * 1 * 2)),
    (B.Q6_G32, B.LAYOUT_CANONICAL, 1, 7, 64, (7 * 64 * 6 // 8, 7 * 2 * 2)),
    (B.F16, B.LAYOUT_DEVICE, 1, 65, 64, (128 * 64 * 2, 0)),
    (B.BF16, B.LAYOUT_CANONICAL, 3, 5, 32, (3 * 5 * 32 * 2, 0)),
])
def test_weight_bytes(fmt, layout, batch, n, k, want):
    assert B.qm_weight_bytes(fmt, layout, batch, n, k) == want


@pytest.mark.parametrize("args,status", [
    ((9, 0, 1, 4, 64), 4),          # bad format
    ((0, 0, 1, 4, 64), 4),          # bad format
    ((1, 7, 1, 4, 64), 5),          # bad layout
    ((1, 0, 1, 4, 48), 2),          # k % 32
    ((1, 0, 0, 4, 64), 2),          # batch 0
])
def test_weight_bytes_errors(args, status):
    with pytest.raises(B.QmError) as e:
        B.qm_weight_bytes(*args)
    assert e.value.status == status
    assert B.qm_last_error()


def _fake_weight(fmt=1, layout=1, batch=1, n=64, k=64, qdata=0x10000, scales=0x20000):
    return B.CQWeight(fmt, layout, batch, n, k, qdata, scales)


def _call(name, *args):
    return getattr(B.lib(), name)(*args)


def test_gemv_validation_before_device_work():
    L = B.lib()
    x, y = ctypes.c_void_p(0x30000), ctypes.c_void_p(0x40000)
    cases = [
        (None, 1),                                          # null descriptor
        (_fake_weight(layout=0), 5),                        # canonical layout
        (_fake_weight(k=48), 2),                            # k % 32
        (_fake_weight(batch=2), 2),                         # batched GEMV
        (_fake_weight(fmt=9), 4),                           # unknown format
        (_fake_weight(qdata=0x10008), 3),                   # misaligned
        (_fake_weight(qdata=0), 1),                         # null codes
    ]
    for w, status in cases:
        st = L.qmatmul_gemv(ctypes.byref(w) if w is not None else None, x, y, None)
        assert st == status, (w and (w.format, w.layout, w.k, w.batch), st)
        assert B.qm_last_error()
    w = _fake_weight()
    assert L.qmatmul_gemv(ctypes.byref(w), ctypes.c_void_p(0x30004), y, None) == 3   # x misaligned
    assert L.qmatmul_gemv(ctypes.byref(w), None, y, None) == 1


def test_gemm_and_moe_validation():
    L = B.lib()
    w = _fake_weight()
    x, y = ctypes.c_void_p(0x30000), ctypes.c_void_p(0x40000)
    assert L.qmatmul_gemm(ctypes.byref(w), x, 0, y, None) == 2          # m = 0
    assert L.qmatmul_gemm(ctypes.byref(w), x, 70000, y, None) == 2      # m too large
    assert L.qmatmul_gemm(ctypes.byref(_fake_weight(fmt=9)), x, 16, y, None) == 4   # unknown format
    for f in (B.F16, B.BF16):                                           # float formats: same checks
        assert L.qmatmul_gemm(ctypes.byref(_fake_weight(fmt=f, layout=0)), x, 16, y, None) == 5
        assert L.qmatmul_gemm(ctypes.byref(_fake_weight(fmt=f)), x, 70000, y, None) == 2
    assert L.qmatmul_gemm(ctypes.byref(_fake_weight(layout=0)), x, 16, y, None) == 5
    p = ctypes.c_void_p(0x50000)
    assert L.qmoe_route(p, 16, 2000, 8, p, p, p, p, p, None) == 2       # too many experts
    assert L.qmoe_route(p, 16, 128, 17, p, p, p, p, p, None) == 2       # top_k > 16
    assert L.qmoe_route(p, 16, 4, 8, p, p, p, p, p, None) == 2          # top_k > E
    assert L.qmoe_route(p, 16, 128, 8, p, p, None, p, p, None) == 1     # null counts
    g = _fake_weight(batch=8, n=96, k=64)
    d = _fake_weight(batch=8, n=64, k=96)
    bad = _fake_weight(batch=8, n=64, k=64)
    ws = ctypes.c_void_p(0x60000)
    args = lambda wg, wu, wd, nbytes, ids=p: L.qmoe_grouped_gemm(
        ctypes.byref(wg), ctypes.byref(wu), ctypes.byref(wd), x, 16, 2, ids, p, p, p, p, y, ws, nbytes, None)
    need = B.qmoe_workspace_bytes(16, 8, 2, 64, 96)
    assert need == 16 * 2 * 96 * 2 + 16 * 2 * 64 * 2              # h and per-assignment outputs, fp16
    assert args(g, g, bad, need) == 2                                  # down shape mismatch
    assert args(g, g, d, need - 1) == 6                                # workspace too small
    g8 = _fake_weight(fmt=2, batch=8, n=96, k=64)
    assert args(g8, g, d, need) == 4                                   # gate, up and down formats differ
    gf, df = _fake_weight(fmt=B.F16, batch=8, n=96, k=64), _fake_weight(fmt=B.F16, batch=8, n=64, k=96)
    assert args(gf, gf, df, need) == 4                                 # float experts are not taken
    assert args(g, g, d, need, ids=None) == 1                          # topk_ids required
    # the allocation-free variant: sizes beyond the library's scratch are
    # refused before anything touches the device
    na = lambda wg, wu, wd, m, ids=p: L.qmoe_grouped_gemm_noalloc(
        ctypes.byref(wg), ctypes.byref(wu), ctypes.byref(wd), x, m, 8, ids, p, p, p, p, y, None)
    g2 = _fake_weight(batch=16, n=768, k=2048)
    d2 = _fake_weight(batch=16, n=2048, k=768)
    assert B.qmoe_workspace_bytes(744, 16, 8, 2048, 768) <= B.NOALLOC_SCRATCH_BYTES
    assert B.qmoe_workspace_bytes(745, 16, 8, 2048, 768) > B.NOALLOC_SCRATCH_BYTES
    assert na(g2, g2, d2, 745) == 6 and "scratch" in B.qm_last_error()
    assert na(g2, g2, d2, 744, ids=None) == 1
    assert na(g2, g2, bad, 16) == 2


def test_quantise_repack_validation():
    L = B.lib()
    w = _fake_weight(layout=1)
    p = ctypes.c_void_p(0x70000)
    assert L.qm_quantise(1, p, ctypes.byref(w), None) == 5            # must write canonical
    wc = _fake_weight(layout=0)
    assert L.qm_quantise(2, p, ctypes.byref(wc), None) == 4           # format mismatch
    assert L.qm_quantise(1, ctypes.c_void_p(0x70004), ctypes.byref(wc), None) == 3
    assert L.qm_repack(ctypes.byref(wc), ctypes.byref(wc), None) == 5  # same layout
    other = _fake_weight(layout=1, n=65)
    assert L.qm_repack(ctypes.byref(wc), ctypes.byref(other), None) == 2


def test_error_text_is_thread_local():
    import threading
    L = B.lib()
    L.qm_weight_bytes(9, 0, 1, 1, 32, ctypes.byref(ctypes.c_size_t()), ctypes.byref(ctypes.c_size_t()))
    main_msg = B.qm_last_error()
    seen = {}

    def other():
        seen["before"] = B.qm_last_error()
        L.qm_weight_bytes(1, 9, 1, 1, 32, ctypes.byref(ctypes.c_size_t()), ctypes.byref(ctypes.c_size_t()))
        seen["after"] = B.qm_last_error()

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen["before"] == ""
    assert "layout" in seen["after"]
    assert B.qm_last_error() == main_msg and "format" in main_msg


def test_float_formats_need_no_scales():
    """F16/BF16 descriptors may carry a null scale pointer; the integer
    formats may not."""
    L = B.lib()
    y = ctypes.c_void_p(0x40000)
    for f in (B.F16, B.BF16):
        w = _fake_weight(fmt=f, layout=0, scales=0)
        # passes the descriptor checks and stops at the null output
        assert L.qm_dequantise(ctypes.byref(w), None, None) == 1
        assert "null output" in B.qm_last_error()
    w = _fake_weight(fmt=B.Q5_G32, layout=0, scales=0)
    assert L.qm_dequantise(ctypes.byref(w), None, None) == 1
    assert "null data pointer" in B.qm_last_error()
    w = _fake_weight(fmt=B.F16, scales=0x20008)                       # misaligned but unused
    assert L.qmatmul_gemv(ctypes.byref(w), ctypes.c_void_p(0x30004), y, None) == 3   # x still checked


def test_gemv_swiglu_validation():
    L = B.lib()
    x, h = ctypes.c_void_p(0x30000), ctypes.c_void_p(0x40000)
    w = _fake_weight()
    call = lambda g, u, xp=x, hp=h: L.qmatmul_gemv_swiglu(ctypes.byref(g), ctypes.byref(u), xp, hp, None)
    assert L.qmatmul_gemv_swiglu(None, ctypes.byref(w), x, h, None) == 1        # null descriptor
    assert call(w, _fake_weight(fmt=2)) == 4                                     # formats differ
    assert call(w, _fake_weight(n=65)) == 2                                      # n differs
    assert call(w, _fake_weight(k=96)) == 2                                      # k differs
    assert call(w, _fake_weight(layout=0)) == 5                                  # not DEVICE layout
    assert call(w, _fake_weight(batch=2)) == 2                                   # batch != 1
    assert call(w, w, xp=ctypes.c_void_p(0x30004)) == 3                          # x misaligned
    assert call(w, w, hp=ctypes.c_void_p(0x40002)) == 3                          # h misaligned
    assert call(w, w, xp=None) == 1                                              # null x
    assert B.qm_last_error()


def test_gemv_grouped_validation():
    L = B.lib()
    x0, y0 = 0x30000, 0x40000

    def call(ws, xs=None, ys=None, count=None):
        n = len(ws)
        descs = (B.CQWeight * max(n, 1))(*ws)
        xs = xs if xs is not None else [x0] * n
        ys = ys if ys is not None else [y0 + 0x1000 * i for i in range(n)]
        xp = (ctypes.c_void_p * max(n, 1))(*xs)
        yp = (ctypes.c_void_p * max(n, 1))(*ys)
        return L.qmatmul_gemv_grouped(n if count is None else count, descs, xp, yp, None)

    w = _fake_weight()
    assert call([w], count=0) == 2                                     # count < 1
    assert call([w] * 9) == 2                                          # count > 8
    assert L.qmatmul_gemv_grouped(1, None, None, None, None) == 1      # null arrays
    assert call([w, _fake_weight(fmt=2)]) == 4                         # formats differ
    assert call([w, _fake_weight(k=96)]) == 2                          # k differs
    assert call([w, _fake_weight(layout=0)]) == 5                      # not DEVICE layout
    assert call([w, _fake_weight(batch=2)]) == 2                       # batch != 1
    assert call([w, w], xs=[x0, x0 + 4]) == 3                          # x[1] misaligned
    assert call([w, w], ys=[y0, y0 + 2]) == 3                          # y[1] misaligned
    assert call([w, w], xs=[x0, 0]) == 1                               # null x[1]
    assert B.qm_last_error()


def test_gemm_grouped_validation():
    L = B.lib()
    x = ctypes.c_void_p(0x30000)

    def call(ws, ys=None, m=16, xp=x, count=None):
        n = len(ws)
        descs = (B.CQWeight * max(n, 1))(*ws)
        ys = ys if ys is not None else [0x40000 + 0x1000 * i for i in range(n)]
        yp = (ctypes.c_void_p * max(n, 1))(*ys)
        return L.qmatmul_gemm_grouped(n if count is None else count, descs, xp, m, yp, None)

    w = _fake_weight()
    assert call([w], count=0) == 2                                     # count < 1
    assert call([w] * 5) == 2                                          # count > 4
    assert L.qmatmul_gemm_grouped(1, None, x, 16, None, None) == 1     # null arrays
    assert call([w], m=0) == 2                                         # m < 1
    assert call([w, _fake_weight(fmt=2)]) == 4                         # formats differ
    assert call([_fake_weight(fmt=9)] * 2) == 4                        # unknown format
    assert call([_fake_weight(fmt=B.BF16), _fake_weight(fmt=B.F16)]) == 4   # float formats differ
    assert call([w, _fake_weight(k=96)]) == 2                          # k differs
    assert call([w, _fake_weight(layout=0)]) == 5                      # not DEVICE layout
    assert call([w, w], ys=[0x40000, 0x40002]) == 3                    # y[1] misaligned
    assert call([w], xp=ctypes.c_void_p(0x30004)) == 3                 # x misaligned
    assert call([w], xp=None) == 1                                     # null x
    assert B.qm_last_error()


def test_attention_decode_validation():
    L = B.lib()
    p = ctypes.c_void_p(0x50000)
    ws = ctypes.c_void_p(0x60000)
    need = B.qattn_decode_workspace_bytes(16, 128)
    assert need == 16 * 256 * 130 * 4
    call = lambda hq=16, hkv=8, d=128, n=100, mx=4096, scale=0.088, q=p, o=p, w=ws, nb=need: \
        L.qattn_decode(q, p, p, hq, hkv, d, n, mx, scale, o, w, nb, None)
    assert call(d=96) == 2                       # head_dim
    assert call(hq=12, hkv=8) == 2               # not a multiple
    assert call(hq=72, hkv=8) == 2               # more than 8 query heads per KV head
    assert call(n=0) == 2 and call(n=5000) == 2  # len outside [1, max_len]
    assert call(mx=300000, n=10) == 2            # max_len too large
    assert call(scale=float("inf")) == 1
    assert call(q=None) == 1
    assert call(q=ctypes.c_void_p(0x50008)) == 3
    assert call(nb=need - 1) == 6
    assert call(w=None) == 6
    with pytest.raises(B.QmError):
        B.qattn_decode_workspace_bytes(16, 80)
    assert B.qm_last_error()


def test_attention_prefill_validation():
    L = B.lib()
    p = ctypes.c_void_p(0x50000)
    call = lambda hq=32, hkv=8, d=64, m=128, p0=0, mx=4096, scale=0.125, q=p, o=p, w=None: \
        L.qattn_prefill(q, p, p, hq, hkv, d, m, p0, mx, scale, o, w, 1 << 20, None)
    assert call(d=80) == 2
    assert call(hq=12, hkv=8) == 2
    assert call(m=0) == 2 and call(m=70000, mx=200000) == 2
    assert call(p0=4000, m=128) == 2               # past max_len
    assert call(p0=-1) == 2
    assert call(scale=float("nan")) == 1 and call(scale=-0.5) == 1 and call(scale=0.0) == 1
    assert call(o=None) == 1
    assert call(w=ctypes.c_void_p(0x60008)) == 3                     # workspace alignment
    assert call(o=ctypes.c_void_p(0x50004)) == 3                     # output alignment
    rows = lambda out=p, d=64: L.qattn_prefill_rows_f16(p, p, p, 32, 8, d, 128, 0, 4096, 0.125, out, None, 0, None)
    assert rows(out=None) == 1 and rows(d=80) == 2 and rows(out=ctypes.c_void_p(0x50008)) == 3
    nb = ctypes.c_size_t()
    assert L.qattn_prefill_workspace_bytes(32, 80, 128, 0, ctypes.byref(nb)) == 2
    assert L.qattn_prefill_workspace_bytes(32, 64, 0, 0, ctypes.byref(nb)) == 2
    assert L.qattn_prefill_workspace_bytes(32, 64, 128, 0, None) == 1
    assert call(q=ctypes.c_void_p(0x50004)) == 3
    assert B.qm_last_error()


def test_decode_glue_validation():
    """Every call stops at argument validation (none reaches a launch)."""
    L = B.lib()
    p = ctypes.c_void_p(0x50000)
    odd = ctypes.c_void_p(0x50001)
    emb = lambda vocab=1000, hidden=256, t=p, tab=p, x=p: L.qdec_embed(tab, vocab, hidden, t, x, None)
    assert emb(vocab=0) == 2 and emb(hidden=0) == 2 and emb(vocab=1 << 31) == 2
    assert emb(t=None) == 1 and emb(tab=odd) == 3 and emb(x=ctypes.c_void_p(0x50002)) == 3
    norm = lambda rows=1, hidden=256, eps=1e-6, x=p, r=None, w=p, o=p: L.qdec_rmsnorm(x, r, w, rows, hidden, eps, o, None)
    assert norm(rows=-1) == 2 and norm(hidden=0) == 2 and norm(rows=70000) == 2
    assert norm(eps=-1.0) == 1 and norm(eps=float("nan")) == 1 and norm(eps=float("inf")) == 1
    assert norm(w=None) == 1 and norm(o=None) == 1
    assert norm(w=odd) == 3 and norm(r=ctypes.c_void_p(0x50002)) == 3
    rope = lambda hq=4, hkv=2, d=64, pos=0, mx=128, theta=1e4, q=p, kc=p, qn=None, kn=None, tab=None, tl=0: \
        L.qdec_rope_append(q, p, p, hq, hkv, d, pos, mx, theta, qn, kn, 1e-6, tab, tl, p, kc, p, None)
    assert rope(qn=p) == 1 and rope(qn=p, kn=ctypes.c_void_p(0x50001)) == 1
    assert rope(d=96) == 2 and rope(hq=0) == 2 and rope(hkv=2000) == 2
    assert rope(pos=128) == 2 and rope(pos=-1) == 2 and rope(mx=300000, pos=5) == 2
    assert rope(theta=1.0) == 1 and rope(theta=float("nan")) == 1
    assert rope(q=None) == 1 and rope(kc=odd) == 3
    assert rope(pos=7, tab=p, tl=7) == 1 and rope(tab=ctypes.c_void_p(0x50004), tl=8) == 1   # table too short / misaligned
    assert L.qdec_cast_f16(p, -1, p, None) == 2 and L.qdec_cast_f16(None, 4, p, None) == 1
    assert L.qdec_cast_f16(ctypes.c_void_p(0x50002), 4, p, None) == 3
    am = lambda n=4, x=p, t=p, w=p, nb=2048: L.qdec_argmax(x, n, t, w, nb, None)
    assert am(n=0) == 2 and am(x=None) == 1 and am(t=odd) == 3 and am(w=odd) == 3
    assert am(nb=2047) == 6 and am(w=None) == 6
    assert B.qm_last_error()


def test_argmax_workspace_constant_matches_header():
    import re
    hdr = open(os.path.join(os.path.dirname(__file__), "..", "include", "qmatmul.h")).read()
    assert int(re.search(r"#define QDEC_ARGMAX_WORKSPACE_BYTES (\d+)", hdr).group(1)) == B.ARGMAX_WORKSPACE_BYTES


def test_fp16_output_variants_validation():
    L = B.lib()
    p = ctypes.c_void_p(0x50000)
    need = B.qattn_decode_workspace_bytes(16, 128)
    call = lambda o=p, d=128, n=10: L.qattn_decode_f16(p, p, p, 16, 8, d, n, 64, 0.1, o, p, need, None)
    assert call(o=None) == 1 and call(o=ctypes.c_void_p(0x50001)) == 3 and call(d=80) == 2 and call(n=65) == 2
    w = B.empty_qweight(B.Q4_G32, B.LAYOUT_DEVICE, 1, 64, 64, device="cpu")
    assert L.qmatmul_gemv_swiglu_f16(ctypes.byref(w.c()), ctypes.byref(w.c()), p, None, None) == 1
    assert L.qmatmul_gemv_swiglu_f16(ctypes.byref(w.c()), ctypes.byref(w.c()), p, ctypes.c_void_p(0x50001),
                                     None) == 3
    assert B.qm_last_error()


def test_fused_rmsnorm_gemv_validation():
    L = B.lib()
    p = ctypes.c_void_p(0x50000)
    w = B.empty_qweight(B.Q4_G32, B.LAYOUT_DEVICE, 1, 64, 1024, device="cpu")
    descs = (B.CQWeight * 1)(w.c())
    ys = (ctypes.c_void_p * 1)(0x70000)
    call = lambda x=p, r=None, g=p, eps=1e-6, xo=ctypes.c_void_p(0x90000), d=descs, n=1: \
        L.qmatmul_gemv_grouped_rmsnorm(n, d, x, r, g, eps, xo, ys, None)
    assert call(n=0) == 2 and call(n=9) == 2
    assert call(x=None) == 1 and call(xo=None) == 1 and call(g=None) == 1
    assert call(eps=-1.0) == 1
    assert call(x=ctypes.c_void_p(0x50004)) == 3 and call(g=ctypes.c_void_p(0x50002)) == 3
    assert call(xo=ctypes.c_void_p(0x50000 + 2048)) == 1          # overlaps x
    big = B.empty_qweight(B.Q4_G32, B.LAYOUT_DEVICE, 1, 64, 8192, device="cpu")
    assert call(d=(B.CQWeight * 1)(big.c())) == 2                  # k > 4096
    q2 = B.empty_qweight(B.Q2_G32, B.LAYOUT_DEVICE, 1, 64, 1024, device="cpu")
    two_ys = (ctypes.c_void_p * 2)(0x70000, 0x78000)
    mixed = L.qmatmul_gemv_grouped_rmsnorm(2, (B.CQWeight * 2)(w.c(), q2.c()), p, None, p, 1e-6,
                                           ctypes.c_void_p(0x90000), two_ys, None)
    assert mixed == 4                                              # one format per call
    sw = lambda h=p, xo=ctypes.c_void_p(0x90000): L.qmatmul_gemv_swiglu_rmsnorm_f16(
        ctypes.byref(w.c()), ctypes.byref(w.c()), p, None, p, 1e-6, xo, h, None)
    assert sw(h=None) == 1 and sw(h=ctypes.c_void_p(0x50001)) == 3 and sw(xo=p) == 1
    assert B.qm_last_error()


def test_qkv_rope_epilogue_validation():
    L = B.lib()
    p = ctypes.c_void_p(0x50000)
    wq = B.empty_qweight(B.Q4_G32, B.LAYOUT_DEVICE, 1, 256, 256, device="cpu")
    wk = B.empty_qweight(B.Q4_G32, B.LAYOUT_DEVICE, 1, 128, 256, device="cpu")
    good = (B.CQWeight * 3)(wq.c(), wk.c(), wk.c())
    bad = (B.CQWeight * 3)(wq.c(), wq.c(), wk.c())
    call = lambda w=good, d=64, pos=3, mx=16, tab=p, qo=p, xo=ctypes.c_void_p(0x90000): \
        L.qmatmul_gemv_qkv_rmsnorm_rope(w, p, None, p, 1e-6, xo, 4, 2, d, pos, mx, tab, qo, p, p, None)
    assert call(w=bad) == 2                       # k rows != n_kv_heads * head_dim
    assert call(d=96) == 2 and call(pos=16) == 2 and call(pos=-1) == 2
    assert call(tab=None) == 1 and call(qo=None) == 1 and call(xo=p) == 1
    assert call(tab=ctypes.c_void_p(0x50004)) == 3
    assert L.qdec_rope_table(0, 64, 1e4, p, None) == 2 and L.qdec_rope_table(8, 80, 1e4, p, None) == 2
    assert L.qdec_rope_table(8, 64, 1.0, p, None) == 1 and L.qdec_rope_table(8, 64, 1e4, None, None) == 1
    assert L.qdec_rope_table(8, 64, 1e4, ctypes.c_void_p(0x50004), None) == 3
    rt3 = lambda n=8, d=64, theta=5e5, f=32.0, lo=1.0, hi=4.0, orig=8192.0, t=p: \
        L.qdec_rope_table_llama3(n, d, theta, f, lo, hi, orig, t, None)
    assert rt3(n=0) == 2 and rt3(d=96) == 2 and rt3(n=300000) == 2
    assert rt3(theta=1.0) == 1 and rt3(f=0.5) == 1 and rt3(f=float("inf")) == 1 and rt3(f=float("nan")) == 1
    assert rt3(lo=0.0) == 1 and rt3(hi=1.0) == 1 and rt3(hi=float("inf")) == 1 and rt3(orig=0.0) == 1
    assert rt3(orig=float("nan")) == 1 and rt3(t=None) == 1 and rt3(t=ctypes.c_void_p(0x50004)) == 3
    assert B.qm_last_error()


def test_prefill_glue_validation():
    L = B.lib()
    p = ctypes.c_void_p(0x50000)
    assert L.qdec_embed_rows(p, 100, 64, p, 40000, p, None) == 2 and L.qdec_embed_rows(p, 0, 64, p, 4, p, None) == 2
    assert L.qdec_embed_rows(None, 100, 64, p, 4, p, None) == 1
    rr = lambda d=64, m=8, p0=0, mx=64, il=0, theta=1e4, qo=p, kn=None, tab=None, tl=0: L.qdec_rope_append_rows(
        p, p, p, 4, 2, d, m, p0, mx, theta, il, None, kn, 1e-6, tab, tl, qo, p, p, None)
    assert rr(kn=p) == 1
    assert rr(tab=p, tl=7) == 1 and rr(tab=ctypes.c_void_p(0x50004), tl=64) == 1   # table too short / misaligned
    assert rr(d=80) == 2 and rr(m=0) == 2 and rr(p0=60) == 2 and rr(il=2) == 1 and rr(theta=0.5) == 1
    assert rr(qo=None) == 1 and rr(qo=ctypes.c_void_p(0x50001)) == 3
    assert L.qdec_heads_to_rows_f16(p, 0, 4, 64, p, None) == 2 and L.qdec_heads_to_rows_f16(None, 4, 4, 64, p, None) == 1
    assert L.qdec_swiglu_f16(p, p, -1, p, None) == 2 and L.qdec_swiglu_f16(None, p, 4, p, None) == 1
    assert L.qdec_swiglu_f16(p, p, 4, ctypes.c_void_p(0x50001), None) == 3
    assert B.qm_last_error()
