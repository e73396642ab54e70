"""Pins of the CPU oracle against facts fixed outside it.

Each check below is chosen so that a plausible slip in the oracle (a dropped
term, a wrong sign or index, a transposed operand, the wrong rounding mode,
the wrong branch of the SwiGLU) fails at least one of them:

* IEEE fp16 rounding against Python's own half-precision packer (``struct``),
* hand-derived quantisation / packing / routing examples (tests/golden),
* exhaustive dequantisation against exact rational products,
* GEMV / GEMM against exact rational brute force, integer grids with
  closed-form answers and one-hot inputs,
* routing against an independent repeated-argmax selection and the softmax's
  closed-form ratios, bucketing against Python's stable ``sorted``,
* the MoE layer against dense evaluation, a top-1 special case, identical
  experts and a hand-computed scalar example; SiLU against its identities,
* RoPE angles of every pair against hand values, the Llama 3 frequency rule
  by its regimes, band edges and blend, and one-layer decode steps
  whose residuals, norms, SwiGLU branch and per-head q/k norms have
  written-out closed forms.
"""

import math
import os
import struct
from fractions import Fraction

import numpy as np
import pytest

from oracle import qmatmul_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.txt")
FMT_NAMES = {"Q2": O.Q2, "Q3": O.Q3, "Q4": O.Q4, "Q5": O.Q5, "Q6": O.Q6, "Q8": O.Q8}
INT_FMTS = [O.Q2, O.Q3, O.Q4, O.Q5, O.Q6, O.Q8]


def _half_bits_struct(x: float) -> int:
    return struct.unpack("<H", struct.pack("<e", x))[0]


def _half_value_struct(bits: int) -> float:
    return struct.unpack("<e", struct.pack("<H", bits))[0]


def _golden_lines(kind):
    out = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.split()[0] == kind:
                out.append([p.strip() for p in line.split("|")])
    return out


# --------------------------------------------------------------- fp16 rounding

def test_fp16_rounding_matches_struct_packer():
    rng = np.random.default_rng(1)
    vals = np.concatenate([
        rng.standard_normal(4000).astype(np.float32) * 0.01,
        rng.standard_normal(2000).astype(np.float32) * 1e-6,        # subnormal fp16
        np.array([0.0, 65504.0, 6.1035156e-05, 5.9604645e-08, 2.9802322e-08,
                  1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11], dtype=np.float32),  # ties
    ])
    got = O.fp16_bits(vals)
    want = np.array([_half_bits_struct(float(v)) for v in vals], dtype=np.uint16)
    assert np.array_equal(got, want)
    # values back
    assert np.array_equal(O.fp16_value(want),
                          np.array([_half_value_struct(int(b)) for b in want], dtype=np.float32))


# ------------------------------------------------------------- worked examples

@pytest.mark.parametrize("row", _golden_lines("quant"))
def test_quantise_worked_examples(row):
    head, w_s, s_hex, q_s, dq_s = row
    fmt = FMT_NAMES[head.split()[1]]
    wv = [float(t) for t in w_s.split()]
    w = np.zeros((1, 32), np.float32)
    w[0, :len(wv)] = wv
    q, s16 = O.quantise(w, fmt)
    qv = [int(t) for t in q_s.split()]
    assert s16.shape == (1, 1) and int(s16[0, 0]) == int(s_hex, 16)
    assert q[0, :len(qv)].tolist() == qv
    assert not q[0, len(qv):].any()
    if dq_s != "-":
        dq = O.dequantise(O.pack(q, fmt), s16, fmt)
        want = [float(t) for t in dq_s.split()]
        assert dq[0, :len(want)].tolist() == want


@pytest.mark.parametrize("row", _golden_lines("pack"))
def test_pack_worked_example(row):
    fmt = FMT_NAMES[row[0].split()[1]]
    codes = [int(t) for t in row[1].split()]
    q = np.zeros((1, 32), np.int8)
    q[0, :len(codes)] = codes
    want = [int(t, 16) for t in row[2].split()]
    b = O.pack(q, fmt)
    assert b.shape == (1, 4 * O.BITS[fmt])
    assert b[0, :len(want)].tolist() == want and not b[0, len(want):].any()
    assert O.unpack(b, fmt).tolist() == q.tolist()


def test_route_and_bucket_worked_example():
    (row,) = _golden_lines("route")
    e, k = (int(t) for t in row[0].split()[1:3])
    logits = np.array([[float(t) for t in r.split()] for r in row[1].split(";")], np.float32)
    ids, gates = O.moe_route(logits, k)
    assert ids.tolist() == [[int(t) for t in r.split()] for r in row[2].split(";")]
    want_g = np.array([[float(t) for t in r.split()] for r in row[3].split(";")])
    assert np.allclose(gates, want_g, rtol=0, atol=1e-15)
    (b,) = _golden_lines("bucket")
    counts, offsets, srt = O.moe_bucket(ids, e)
    assert counts.tolist() == [int(t) for t in b[2].split()[1:]]
    assert offsets.tolist() == [int(t) for t in b[3].split()[1:]]
    assert srt.tolist() == [int(t) for t in b[4].split()[1:]]


# ------------------------------------------------------------------ invariants

@pytest.mark.parametrize("fmt", INT_FMTS)
def test_quantise_invariants_random_groups(fmt):
    rng = np.random.default_rng(7 + fmt)
    w = (rng.standard_normal((625, 1024)).astype(np.float32) * np.float32(0.02))
    q, s16 = O.quantise(w, fmt)
    s = O.fp16_value(s16).astype(np.float64)
    qg = q.reshape(625, 32, 32).astype(np.int64)
    # every normal-range group reaches +-qmax exactly and never -8 for Q4
    assert np.all(np.abs(qg).max(axis=2) == O.QMAX[fmt])
    assert q.min() >= -O.QMAX[fmt]
    # reconstruction error within half a step (plus the fp32 division's rounding)
    dq = O.dequantise(O.pack(q, fmt), s16, fmt).astype(np.float64)
    err = np.abs(dq - w.astype(np.float64)).reshape(625, 32, 32)
    assert np.all(err <= (s[:, :, None] / 2) * (1 + 2.0 ** -20))
    # re-quantising the dequantised matrix reproduces the codes and scales
    q2, s2 = O.quantise(dq.astype(np.float32), fmt)
    assert np.array_equal(q2, q) and np.array_equal(s2, s16)


def test_quantise_scale_is_fp16_of_fp32_quotient():
    """Scale = fp16_RNE(fp32(max|w| / qmax)), checked with Python floats:
    the fp32 quotient is the double quotient rounded once to fp32."""
    rng = np.random.default_rng(3)
    w = rng.standard_normal((64, 64)).astype(np.float32) * np.float32(0.02)
    for fmt in INT_FMTS:
        _, s16 = O.quantise(w, fmt)
        for n in range(64):
            for g in range(2):
                m = max(abs(float(v)) for v in w[n, 32 * g:32 * g + 32])
                q32 = struct.unpack("<f", struct.pack("<f", m / O.QMAX[fmt]))[0]
                assert int(s16[n, g]) == _half_bits_struct(q32)


@pytest.mark.parametrize("fmt", INT_FMTS)
def test_pack_roundtrip_all_codes(fmt):
    lo, hi = O.QLO[fmt], O.QHI[fmt]
    codes = np.arange(lo, hi + 1)
    rng = np.random.default_rng(11)
    q = rng.choice(codes, size=(37, 256)).astype(np.int8)
    b = O.pack(q, fmt)
    assert b.shape == (37, 256 * O.BITS[fmt] // 8)
    assert np.array_equal(O.unpack(b, fmt), q)


@pytest.mark.parametrize("fmt", INT_FMTS)
def test_pack_bit_by_bit(fmt):
    """Every code's bits at their stream positions, read back one bit at a
    time with Python integers (little-endian stream)."""
    rng = np.random.default_rng(31 + fmt)
    nb = O.BITS[fmt]
    q = rng.integers(O.QLO[fmt], O.QHI[fmt] + 1, size=(3, 64)).astype(np.int8)
    b = O.pack(q, fmt)
    for r in range(3):
        stream = int.from_bytes(bytes(b[r].tolist()), "little")
        for kk in range(64):
            field = (stream >> (nb * kk)) & ((1 << nb) - 1)
            assert field == int(q[r, kk]) % (1 << nb)


@pytest.mark.parametrize("fmt", INT_FMTS)
def test_dequantise_exhaustive_against_exact_products(fmt):
    lo, hi = O.QLO[fmt], O.QHI[fmt]
    codes = list(range(lo, hi + 1))
    scale_bits = [0x0000, 0x0001, 0x0002, 0x03FF, 0x0400, 0x1C63, 0x1DDA, 0x0D29,
                  0x2E66, 0x3C00, 0x5140, 0x7BFF]
    n = len(scale_bits)
    reps = -(-32 // len(codes))
    row = (codes * reps)[:32] if len(codes) < 32 else codes
    k = (len(row) + 31) // 32 * 32
    q = np.zeros((n, k), np.int8)
    for i in range(n):
        q[i, :len(row)] = row
    s16 = np.array([[b] * (k // 32) for b in scale_bits], np.uint16)
    dq = O.dequantise(O.pack(q, fmt), s16, fmt)
    for i, bits in enumerate(scale_bits):
        sv = Fraction(_half_value_struct(bits))
        for kk in range(k):
            assert Fraction(float(dq[i, kk])) == sv * int(q[i, kk])


def test_f16_tile_value_is_one_rounding_of_exact_product():
    q = np.zeros((1, 32), np.int8)
    q[0, 0] = 7
    s16 = np.array([[0x1DDA]], np.uint16)    # s = 0.00571441650390625
    bits = O.dequantise_f16_tile_value(O.pack(q, O.Q4), s16, O.Q4)
    # exact 7*s = 0.04000091552734375 is not an fp16; nearest fp16 is 0.0400085...
    assert int(bits[0, 0]) == _half_bits_struct(0.04000091552734375)
    assert _half_value_struct(int(bits[0, 0])) != 0.04000091552734375


# ---------------------------------------------------------- float formats

def _bf16_nearest_exact(x: float) -> int:
    """bf16 pattern nearest to x by exact rational comparison of the two
    bf16 neighbours (truncation and the next pattern), ties to even."""
    bits = struct.unpack("<I", struct.pack("<f", x))[0]
    lo = bits >> 16
    cand = [lo, lo + 1]
    vals = [Fraction(struct.unpack("<f", struct.pack("<I", c << 16))[0]) for c in cand]
    d = [abs(v - Fraction(x)) for v in vals]
    if d[0] != d[1]:
        return cand[0] if d[0] < d[1] else cand[1]
    return cand[0] if cand[0] % 2 == 0 else cand[1]


def test_bf16_rounding_hand_values_and_exact_neighbours():
    f = lambda b: struct.unpack("<f", struct.pack("<I", b))[0]
    hand = {0x3F800000: 0x3F80,          # 1.0
            0x3F808000: 0x3F80,          # 1 + 2^-8: tie, keep even 0x3F80
            0x3F818000: 0x3F82,          # 1 + 3*2^-8: tie, odd 0x3F81 rounds up
            0x3F808001: 0x3F81,          # just above the tie
            0xC0200000: 0xC020,          # -2.5
            0x3CA3D70A: 0x3CA4,          # fp32(0.02): lower half 0xD70A > 0x8000
            0x00000001: 0x0000}          # smallest fp32 subnormal
    x = np.array([f(b) for b in hand], np.float32)
    assert O.bf16_bits(x).tolist() == list(hand.values())
    rng = np.random.default_rng(17)
    vals = np.concatenate([rng.standard_normal(3000).astype(np.float32) * 0.02,
                           rng.standard_normal(500).astype(np.float32) * 1e30,
                           rng.standard_normal(500).astype(np.float32) * 1e-38])
    got = O.bf16_bits(vals)
    assert got.tolist() == [_bf16_nearest_exact(float(v)) for v in vals]
    assert np.array_equal(O.bf16_value(got).view(np.uint32), got.astype(np.uint32) << 16)


@pytest.mark.parametrize("fmt", [O.F16, O.BF16])
def test_float_formats_quantise_is_one_rounding(fmt):
    rng = np.random.default_rng(23)
    w = rng.standard_normal((9, 64)).astype(np.float32) * np.float32(0.02)
    bits, s = O.quantise(w, fmt)
    assert s is None and bits.dtype == np.uint16
    want = (O.fp16_bits(w) if fmt == O.F16 else np.vectorize(_bf16_nearest_exact)(w.astype(np.float64)))
    assert np.array_equal(bits, want)
    dq = O.dequantise(O.pack(bits, fmt), None, fmt)
    assert np.array_equal(O.quantise(dq, fmt)[0], bits)              # idempotent
    rel = 2.0 ** -11 if fmt == O.F16 else 2.0 ** -8
    assert np.all(np.abs(dq.astype(np.float64) - w) <= rel * np.abs(w) + 2.0 ** -25)


# ------------------------------------------------------------------ GEMV/GEMM

def _exact_decode(qbytes, s16, fmt, n, k):
    """Independent pure-Python decode of the canonical bytes into Fractions
    (F16 through struct's half-precision unpacker, BF16 as the upper half of
    an fp32 pattern)."""
    rows = []
    for r in range(n):
        row = []
        if fmt in O.FLOATS:
            for kk in range(k):
                bits = int(qbytes[r, kk])
                v = (_half_value_struct(bits) if fmt == O.F16
                     else struct.unpack("<f", struct.pack("<I", bits << 16))[0])
                row.append(Fraction(v))
            rows.append(row)
            continue
        nb = O.BITS[fmt]
        stream = int.from_bytes(bytes(qbytes[r].tolist()), "little")
        for kk in range(k):
            field = (stream >> (nb * kk)) & ((1 << nb) - 1)
            code = field - (1 << nb) if field >= (1 << (nb - 1)) else field
            row.append(Fraction(_half_value_struct(int(s16[r, kk // 32]))) * code)
        rows.append(row)
    return rows


@pytest.mark.parametrize("fmt", INT_FMTS + [O.F16, O.BF16])
def test_gemv_gemm_against_exact_rationals(fmt):
    rng = np.random.default_rng(21 + fmt)
    n, k, m = 5, 96, 3                            # non-square: catches a transpose
    w = rng.standard_normal((n, k)).astype(np.float32) * np.float32(0.02)
    q, s16 = O.quantise(w, fmt)
    qb = O.pack(q, fmt)
    x = rng.standard_normal((m, k)).astype(np.float16)
    wf = _exact_decode(qb, s16, fmt, n, k)
    xf = [[Fraction(float(v)) for v in row] for row in x]
    exact = [[sum(wf[j][kk] * xf[i][kk] for kk in range(k)) for j in range(n)] for i in range(m)]
    y = O.gemm(qb, s16, fmt, x)
    assert y.shape == (m, n)
    for i in range(m):
        yv = O.gemv(qb, s16, fmt, x[i])
        for j in range(n):
            e = float(exact[i][j])
            assert abs(y[i, j] - e) <= 1e-14 * max(1.0, abs(e))
            assert abs(yv[j] - e) <= 1e-14 * max(1.0, abs(e))


@pytest.mark.parametrize("fmt", INT_FMTS)
def test_gemv_integer_grid_is_exact(fmt):
    """Integer weights with a +-qmax in every group quantise with scale 1, so
    y is the exact integer sum (computed here with Python ints)."""
    rng = np.random.default_rng(5)
    qm = O.QMAX[fmt]
    n, k = 48, 160
    wi = rng.integers(-qm, qm + 1, size=(n, k))
    wi[:, ::32] = qm * rng.choice([-1, 1], size=(n, k // 32))
    q, s16 = O.quantise(wi.astype(np.float32), fmt)
    assert np.all(s16 == 0x3C00) and np.array_equal(q, wi)
    xi = rng.integers(-4, 5, size=(3, k))
    y = O.gemm(O.pack(q, fmt), s16, fmt, xi.astype(np.float16))
    want = [[sum(int(wi[j, kk]) * int(xi[i, kk]) for kk in range(k)) for j in range(n)] for i in range(3)]
    assert y.tolist() == want


def test_gemv_one_hot_returns_dequantised_column():
    rng = np.random.default_rng(9)
    w = rng.standard_normal((70, 128)).astype(np.float32) * np.float32(0.02)
    q, s16 = O.quantise(w, O.Q4)
    qb = O.pack(q, O.Q4)
    dq = O.dequantise(qb, s16, O.Q4)
    for kk in (0, 31, 32, 77, 127):
        x = np.zeros(128, np.float16)
        x[kk] = 1.0
        assert np.array_equal(O.gemv(qb, s16, O.Q4, x), dq[:, kk].astype(np.float64))


# ------------------------------------------------------------------------ MoE

def test_route_matches_repeated_argmax_and_softmax_ratios():
    rng = np.random.default_rng(13)
    logits = rng.standard_normal((64, 128)).astype(np.float32)
    logits[:8, 5] = logits[:8, 9] = 3.0            # forced ties inside the top set
    logits[8, :] = 0.0                              # all equal
    ids, gates = O.moe_route(logits, 8)
    for t in range(64):
        work = logits[t].astype(np.float64).copy()
        pick = []
        for _ in range(8):
            j = int(np.argmax(work))               # first maximum = lower index
            pick.append(j)
            work[j] = -np.inf
        assert ids[t].tolist() == pick
        assert abs(gates[t].sum() - 1.0) < 1e-15
        for a in range(8):
            for b in range(8):
                want = math.exp(float(logits[t, pick[a]]) - float(logits[t, pick[b]]))
                assert abs(gates[t, a] / gates[t, b] - want) <= 1e-13 * want
    assert ids[8].tolist() == list(range(8))


def test_bucket_matches_stable_sorted():
    rng = np.random.default_rng(17)
    for ids in (rng.integers(0, 128, size=(100, 8)),
                np.tile(np.arange(8), (50, 1)),                 # 120 empty experts
                np.full((3, 1), 127)):
        e = 128
        counts, offsets, srt = O.moe_bucket(ids, e)
        flat = ids.reshape(-1).tolist()
        assert counts.tolist() == np.bincount(flat, minlength=e).tolist()
        assert offsets[0] == 0 and offsets[-1] == len(flat)
        assert np.array_equal(np.diff(offsets), counts)
        assert srt.tolist() == sorted(range(len(flat)), key=lambda a: (flat[a], a))


def test_silu_identities():
    z = np.linspace(-30, 30, 601)
    s = O.silu(z)
    assert np.allclose(s - O.silu(-z), z, rtol=0, atol=1e-13)       # silu(z)-silu(-z)=z
    assert O.silu(np.array([0.0]))[0] == 0.0
    assert abs(O.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16


def test_gemv_swiglu_hand_example():
    """x = e_0 over integer-grid weights (scale 1): (Wg x)[n] = Wg[n][0] and
    (Wu x)[n] = Wu[n][0], so h[n] = silu(Wg[n][0]) * Wu[n][0], evaluated here
    with scalar math.exp; and h equals the hidden vector of expert_ffn."""
    rng = np.random.default_rng(29)
    n, k = 48, 64
    wg = rng.integers(-7, 8, size=(n, k)); wg[:, ::32] = 7
    wu = rng.integers(-7, 8, size=(n, k)); wu[:, ::32] = 7
    for fmt in (O.Q4, O.Q8):
        gq, gs = O.quantise(wg.astype(np.float32), fmt)
        uq, us = O.quantise(wu.astype(np.float32), fmt)
        x = np.zeros(k, np.float16)
        x[0] = 1.0
        h = O.gemv_swiglu(O.pack(gq, fmt), gs, O.pack(uq, fmt), us, fmt, x)
        dg = O.dequantise(O.pack(gq, fmt), gs, fmt).astype(np.float64)
        du = O.dequantise(O.pack(uq, fmt), us, fmt).astype(np.float64)
        for i in range(n):
            a, b = float(dg[i, 0]), float(du[i, 0])
            want = a / (1.0 + math.exp(-a)) * b
            assert abs(h[i] - want) <= 1e-13 * max(1.0, abs(want))
        if fmt == O.Q4:
            assert np.array_equal(dg, wg) and np.array_equal(du, wu)        # scale 1: exact grid
        # the same h as inside the SwiGLU expert (y = Wd h with Wd = identity)
        y = O.expert_ffn(x.astype(np.float64)[None], dg, du, np.eye(n))
        assert np.allclose(y[0], h, rtol=1e-15, atol=0)


def _grid_expert(rng, n, k):
    w = rng.integers(-7, 8, size=(n, k))
    w[:, ::32] = 7
    q, s16 = O.quantise(w.astype(np.float32), O.Q4)
    return O.pack(q, O.Q4), s16, w


def test_expert_ffn_hand_example():
    """x = e_0, integer grid weights (scale 1): a_i = Wg[i][0], b_i = Wu[i][0],
    y_n = sum_i Wd[n][i] * silu(a_i) * b_i.  Evaluated with scalar math.exp."""
    rng = np.random.default_rng(23)
    h, inter = 32, 64
    gq, gs, wg = _grid_expert(rng, inter, h)
    uq, us, wu = _grid_expert(rng, inter, h)
    dq_, ds, wd = _grid_expert(rng, h, inter)
    x = np.zeros((1, h), np.float16)
    x[0, 0] = 1.0
    logits = np.zeros((1, 1), np.float32)
    out, *_ = O.moe_layer(x, logits, 1, gq[None], gs[None], uq[None], us[None], dq_[None], ds[None])
    for n in range(h):
        want = 0.0
        for i in range(inter):
            a = float(wg[i, 0])
            want += float(wd[n, i]) * (a / (1.0 + math.exp(-a))) * float(wu[i, 0])
        assert abs(out[0, n] - want) <= 1e-12 * max(1.0, abs(want))


def _random_experts(rng, e, h, inter):
    def mk(n, k):
        w = rng.standard_normal((e, n, k)).astype(np.float32) * np.float32(0.02)
        qs = [O.quantise(w[i], O.Q4) for i in range(e)]
        return np.stack([O.pack(q, O.Q4) for q, _ in qs]), np.stack([s for _, s in qs])
    return mk(inter, h) + mk(inter, h) + mk(h, inter)


def test_moe_layer_equals_dense_gate_evaluation():
    rng = np.random.default_rng(29)
    e, h, inter, m, k = 16, 64, 96, 40, 4
    gq, gs, uq, us, dq_, ds = _random_experts(rng, e, h, inter)
    x = rng.standard_normal((m, h)).astype(np.float16)
    logits = rng.standard_normal((m, e)).astype(np.float32)
    out, ids, gates, *_ = O.moe_layer(x, logits, k, gq, gs, uq, us, dq_, ds)
    # dense: every expert on every token, gate matrix zero off the top-k
    x64 = x.astype(np.float64)
    dense_gate = np.zeros((m, e))
    for t in range(m):
        for j in range(k):
            dense_gate[t, ids[t, j]] = gates[t, j]
    ref = np.zeros((m, h))
    for ex in range(e):
        wg = O.dequantise(gq[ex], gs[ex], O.Q4).astype(np.float64)
        wu = O.dequantise(uq[ex], us[ex], O.Q4).astype(np.float64)
        wd = O.dequantise(dq_[ex], ds[ex], O.Q4).astype(np.float64)
        for t in range(m):
            a = wg @ x64[t]
            b = wu @ x64[t]
            hh = (a / (1 + np.exp(-a))) * b
            ref[t] += dense_gate[t, ex] * (wd @ hh)
    assert np.allclose(out, ref, rtol=0, atol=1e-12 * np.abs(ref).max())


def test_moe_top1_and_identical_experts():
    rng = np.random.default_rng(31)
    e, h, inter, m = 8, 32, 64, 12
    gq, gs, uq, us, dq_, ds = _random_experts(rng, e, h, inter)
    x = rng.standard_normal((m, h)).astype(np.float16)
    logits = rng.standard_normal((m, e)).astype(np.float32)
    out1, ids1, g1, *_ = O.moe_layer(x, logits, 1, gq, gs, uq, us, dq_, ds)
    assert np.all(g1 == 1.0)
    for t in range(m):
        ex = int(np.argmax(logits[t]))
        assert ids1[t, 0] == ex
        single, *_ = O.moe_layer(x[t:t + 1], np.zeros((1, 1), np.float32), 1,
                                 gq[ex:ex + 1], gs[ex:ex + 1], uq[ex:ex + 1], us[ex:ex + 1],
                                 dq_[ex:ex + 1], ds[ex:ex + 1])
        assert np.allclose(out1[t], single[0], rtol=0, atol=1e-14 * np.abs(single).max())
    # identical experts: the gates sum to one, so the layer is that expert's FFN
    rep = lambda a: np.repeat(a[:1], e, axis=0)
    outs, *_ = O.moe_layer(x, logits, 4, rep(gq), rep(gs), rep(uq), rep(us), rep(dq_), rep(ds))
    one, *_ = O.moe_layer(x, np.zeros((m, 1), np.float32), 1, gq[:1], gs[:1], uq[:1], us[:1],
                          dq_[:1], ds[:1])
    assert np.allclose(outs, one, rtol=0, atol=1e-13 * np.abs(one).max())


# ------------------------------------------------------------------ attention

def test_attention_hand_example():
    """Scores ln 3 and 0 give weights 3/4 and 1/4: o = 3/4 v0 + 1/4 v1."""
    q = np.array([[1.0, 0.0]])
    k = np.array([[[math.log(3.0), 5.0], [0.0, 7.0], [9.0, 9.0]]])     # row 2 is past the length
    v = np.array([[[4.0, 0.0], [0.0, 8.0], [100.0, 100.0]]])
    o = O.attention_decode(q, k, v, 2, 1.0)
    assert np.allclose(o, [[3.0, 2.0]], rtol=0, atol=1e-15)
    # causal prefill of the same two rows: row 0 sees only itself
    op = O.attention_prefill(np.array([[[1.0, 0.0], [1.0, 0.0]]]), k[:, :2], v[:, :2], 1.0)
    assert np.allclose(op[0, 0], v[0, 0]) and np.allclose(op[0, 1], [3.0, 2.0], atol=1e-15)


def test_attention_closed_forms_and_gqa_mapping():
    rng = np.random.default_rng(41)
    hkv, tmax, d = 2, 9, 4
    k = rng.standard_normal((hkv, tmax, d))
    v = rng.standard_normal((hkv, tmax, d))
    # length 1: the only value row, whatever the scores
    q = rng.standard_normal((6, d))
    assert np.allclose(O.attention_decode(q, k, v, 1, 0.7), v[np.arange(6) // 3, 0], atol=1e-15)
    # zero query: uniform weights, the mean of the valid rows
    z = np.zeros((6, d))
    o = O.attention_decode(z, k, v, 7, 1.0)
    assert np.allclose(o, v[np.arange(6) // 3, :7].mean(axis=1), atol=1e-14)
    # a dominant key: e^-60 of the rest
    kk = k.copy()
    kk[1, 4] = 30.0 * np.ones(d)
    qq = np.ones((6, d))
    o = O.attention_decode(qq, kk, v, 9, 0.5)
    assert np.allclose(o[3:], v[1, 4], atol=1e-20 + 1e-12)
    # heads 0-2 read KV head 0 and heads 3-5 KV head 1: swapping the KV heads
    # swaps the two halves of the output
    o1 = O.attention_decode(q, k, v, 8, 0.3)
    o2 = O.attention_decode(np.concatenate([q[3:], q[:3]]), k[::-1], v[::-1], 8, 0.3)
    assert np.allclose(o1, np.concatenate([o2[3:], o2[:3]]), atol=1e-14)


def test_attention_against_python_loops():
    """Tiny case with math.exp and plain Python sums."""
    rng = np.random.default_rng(42)
    hq, hkv, t, d = 4, 2, 5, 3
    q = rng.standard_normal((hq, d))
    k = rng.standard_normal((hkv, t + 2, d))
    v = rng.standard_normal((hkv, t + 2, d))
    o = O.attention_decode(q, k, v, t, 0.9)
    for h in range(hq):
        g = h // 2
        sc = [0.9 * sum(q[h][i] * k[g][j][i] for i in range(d)) for j in range(t)]
        w = [math.exp(x) for x in sc]
        tot = sum(w)
        for i in range(d):
            assert abs(o[h][i] - sum(w[j] * v[g][j][i] for j in range(t)) / tot) < 1e-13
    qp = rng.standard_normal((hq, t, d))
    op = O.attention_prefill(qp, k[:, :t], v[:, :t], 0.9)
    for h in range(hq):
        for r in range(t):
            # row r of causal prefill = decode attention over the first r+1 rows
            assert np.allclose(op[h, r], O.attention_decode(qp[:, r], k, v, r + 1, 0.9)[h], atol=1e-14)


def test_attention_prefill_chunk_offset():
    """A chunk at offset p0 equals the last rows of the whole prompt, and
    its row i equals decode attention over the first p0 + i + 1 rows."""
    rng = np.random.default_rng(43)
    hq, hkv, n, d = 4, 2, 11, 3
    q = rng.standard_normal((hq, n, d))
    k = rng.standard_normal((hkv, n, d))
    v = rng.standard_normal((hkv, n, d))
    full = O.attention_prefill(q, k, v, 0.8)
    part = O.attention_prefill(q[:, 6:], k, v, 0.8, p0=6)
    assert np.allclose(part, full[:, 6:], atol=1e-14)
    for i in range(5):
        assert np.allclose(part[:, i], O.attention_decode(q[:, 6 + i], k, v, 7 + i, 0.8), atol=1e-14)


# ---------------------------------------------------------------- decode step

def test_rmsnorm_closed_forms():
    w = np.array([1.0, 2.0, -1.0, 0.5])
    assert np.allclose(O.rmsnorm(np.full(4, 3.0), w, 0.0), w)                 # constant vector -> w
    assert np.allclose(O.rmsnorm(np.array([3.0, 4.0, 0.0, 0.0]), np.ones(4), 0.0),
                       np.array([3.0, 4.0, 0.0, 0.0]) / 2.5)                    # rms = 5 / 2
    assert np.allclose(O.rmsnorm(np.zeros(4), w, 1e-6), 0.0)


def test_rope_position_zero_rotation_and_relative_angle():
    rng = np.random.default_rng(44)
    q = rng.standard_normal((3, 8))
    k = rng.standard_normal((3, 8))
    assert np.allclose(O.rope(q, 0, 10000.0), q)                                 # identity at 0
    assert np.allclose(np.linalg.norm(O.rope(q, 17, 1e6), axis=1), np.linalg.norm(q, axis=1))
    # scores depend on the relative position only
    a = np.sum(O.rope(q, 5, 500.0) * O.rope(k, 2, 500.0), axis=1)
    b = np.sum(O.rope(q, 13, 500.0) * O.rope(k, 10, 500.0), axis=1)
    assert np.allclose(a, b)
    # dimension 0 pairs with D/2, rotating by pos radians (theta^0 = 1)
    e = np.zeros((1, 8)); e[0, 0] = 1.0
    r = O.rope(e, 1, 10000.0)
    assert np.allclose(r[0, [0, 4]], [math.cos(1.0), math.sin(1.0)]) and np.allclose(np.delete(r[0], [0, 4]), 0.0)


def _tiny_model(rng, layers=2, h=64, hq=4, hkv=2, d=16, inter=96, vocab=50):
    mk = lambda *sh: rng.standard_normal(sh) * 0.2
    ly = [dict(wq=mk(hq * d, h), wk=mk(hkv * d, h), wv=mk(hkv * d, h), wo=mk(h, hq * d), wg=mk(inter, h),
               wu=mk(inter, h), wd=mk(h, inter), attn_norm=1 + mk(h), ffn_norm=1 + mk(h)) for _ in range(layers)]
    return dict(emb=mk(vocab, h), layers=ly, norm=1 + mk(h), lm_head=mk(vocab, h), hq=hq, hkv=hkv, d=d,
                eps=1e-6, theta=10000.0)


def test_decode_step_zero_layers_and_first_position():
    """With every projection zero the residual stream is the embedding, so
    the logits are lm_head . fp16(rmsnorm(emb[token])); at position 0 the
    attention output is the (fp16) value row itself."""
    rng = np.random.default_rng(45)
    m = _tiny_model(rng)
    z = dict(m)
    z["layers"] = [dict(l, wo=np.zeros_like(l["wo"]), wd=np.zeros_like(l["wd"])) for l in m["layers"]]
    kc = np.zeros((2, 2, 8, 16)); vc = np.zeros((2, 2, 8, 16))
    lg = O.decode_step(z, 7, 0, kc, vc)
    want = m["lm_head"] @ O.f16(O.rmsnorm(m["emb"][7], m["norm"], 1e-6))
    assert np.allclose(lg, want, atol=1e-12)
    # the cache rows written at position 0 are fp16(W x) (k with RoPE at 0 = identity)
    h = O.f16(O.rmsnorm(m["emb"][7], m["layers"][0]["attn_norm"], 1e-6))
    assert np.allclose(vc[0, :, 0], O.f16((m["layers"][0]["wv"] @ h).reshape(2, 16)))
    assert np.allclose(kc[0, :, 0], O.f16((m["layers"][0]["wk"] @ h).reshape(2, 16)))


def test_decode_step_matches_prefill_attention_of_the_sequence():
    """Running decode steps over a sequence fills the cache so that the last
    step's attention equals causal prefill attention over the same keys."""
    rng = np.random.default_rng(46)
    m = _tiny_model(rng, layers=1)
    kc = np.zeros((1, 2, 8, 16)); vc = np.zeros((1, 2, 8, 16))
    toks = [3, 9, 1, 4, 4]
    for p, t in enumerate(toks):
        O.decode_step(m, t, p, kc, vc)
    assert np.all(kc[0, :, 5:] == 0) and np.all(kc[0, :, :5] != 0)
    # the last step's query at position 4 against keys 0..4 equals row 4 of causal prefill
    ly = m["layers"][0]
    x = np.asarray(m["emb"][toks[-1]], dtype=np.float64)
    q = O.f16(O.rope((ly["wq"] @ O.f16(O.rmsnorm(x, ly["attn_norm"], 1e-6))).reshape(4, 16), 4, 10000.0))
    dec = O.attention_decode(q, kc[0], vc[0], 5, 0.25)
    qp = np.zeros((4, 5, 16)); qp[:, 4] = q
    pre = O.attention_prefill(qp, kc[0, :, :5], vc[0, :, :5], 0.25)
    assert np.allclose(dec, pre[:, 4], atol=1e-14)


def test_greedy_token_ties_nan_and_infinities():
    assert O.greedy_token([0.5, 2.0, 2.0, -1.0]) == 1                 # first of equal maxima
    assert O.greedy_token([np.nan, -np.inf, -np.inf]) == 1           # NaN never chosen
    assert O.greedy_token([np.nan, np.nan]) == 0
    assert O.greedy_token([1.0, np.inf, np.nan, np.inf]) == 1
    assert O.greedy_token([-3.0]) == 0
    z = np.random.default_rng(47).standard_normal(1000)
    assert O.greedy_token(z) == int(np.argmax(z))


def test_decode_step_qk_norm_makes_unit_rms_heads():
    """With unit q/k norm gains every cached key row has RMS 1 (RoPE
    preserves the norm; fp16 rounding aside), whatever W_k's scale; with the
    norms absent the rows keep W_k's scale."""
    rng = np.random.default_rng(48)
    m = _tiny_model(rng, layers=1)
    m["layers"][0]["wk"] = m["layers"][0]["wk"] * 37.0
    kc = np.zeros((1, 2, 8, 16)); vc = np.zeros((1, 2, 8, 16))
    O.decode_step(m, 3, 0, kc, vc)
    assert np.sqrt(np.mean(kc[0, :, 0] ** 2, axis=1)).min() > 3.0
    m["layers"][0]["q_norm"] = np.ones(16)
    m["layers"][0]["k_norm"] = np.ones(16)
    for p in range(3):
        O.decode_step(m, 3 + p, p, kc, vc)
        assert np.allclose(np.sqrt(np.mean(kc[0, :, p] ** 2, axis=1)), 1.0, atol=2e-3)
    # a gain of 2 on both doubles the key rows (eps negligible)
    m2 = dict(m); m2["layers"] = [dict(m["layers"][0], k_norm=np.full(16, 2.0))]
    kc2 = np.zeros_like(kc); vc2 = np.zeros_like(vc)
    O.decode_step(m2, 3, 0, kc2, vc2)
    assert np.allclose(kc2[0, :, 0], 2 * kc[0, :, 0], rtol=2e-3, atol=2e-3)


# ------------------------------------------- RoPE schedule, decode-step halves

def test_rope_frequency_schedule_every_pair():
    """Angle of pair i at position p is p * theta^(-2i/D).  With D = 8 and
    theta = 10^4 that is p * 10^-i: at p = 1 the four pairs turn by 1, 0.1,
    0.01 and 0.001 rad, at p = 3 by 3, 0.3, 0.03 and 0.003 rad.  One-hot
    inputs read off each (cos, sin) and the pairing i <-> i + D/2 directly."""
    d = 8
    for pos in (1, 3):
        for i in range(d // 2):
            a = pos * 10.0 ** (-i)
            e = np.zeros((1, d)); e[0, i] = 1.0
            want = np.zeros(d); want[i] = math.cos(a); want[i + d // 2] = math.sin(a)
            assert np.allclose(O.rope(e, pos, 1e4)[0], want, atol=1e-15), (pos, i)
            e = np.zeros((1, d)); e[0, i + d // 2] = 1.0
            want = np.zeros(d); want[i] = -math.sin(a); want[i + d // 2] = math.cos(a)
            assert np.allclose(O.rope(e, pos, 1e4)[0], want, atol=1e-15), (pos, i)
    # D = 4, theta = 100: angles p and p / 10
    r = O.rope(np.array([[1.0, 1.0, 0.0, 0.0]]), 2, 100.0)[0]
    assert np.allclose(r, [math.cos(2.0), math.cos(0.2), math.sin(2.0), math.sin(0.2)], atol=1e-15)


def test_rope_llama3_frequency_rule():
    """The Llama 3 long-context RoPE rule (factor, low, high, L): wavelengths
    w = 2 pi / f below L / high keep f, above L / low become f / factor, and
    in between the ratio f' / f runs linearly in L / w from 1 / factor (at
    L / w = low) to 1 (at L / w = high).
    D = 8, theta = 10^4: f = 1, 0.1, 0.01, 0.001 (w = 6.28, 62.8, 628, 6283);
    with factor 4, low 1, high 4, L = 1000 the cut-offs are 250 and 1000, so
    pairs 0 and 1 keep 1 and 0.1, pair 3 becomes 0.00025 and pair 2 lies in
    the band."""
    f = O.rope_frequencies(8, 1e4, (4, 1, 4, 1000))
    assert f[0] == 1.0 and abs(f[1] - 0.1) <= 1e-17 and abs(f[3] - 0.00025) <= 1e-19
    assert 0.01 / 4 < f[2] < 0.01
    # no scaling at factor 1, whatever the band edges
    assert np.allclose(O.rope_frequencies(64, 5e5, (1, 1, 4, 8192)), O.rope_frequencies(64, 5e5), rtol=1e-15, atol=0)
    # the band: pick theta so that pair 2's wavelength 2 pi sqrt(theta) gives
    # L / w = 1 (long edge), 1.5, 2.5 (the middle), 3.5, 4 (short edge)
    for lw, ratio in ((1.0, 0.25), (1.5, 0.375), (2.5, (0.25 + 1.0) / 2), (3.5, 0.875), (4.0, 1.0)):
        theta = (1000.0 / lw / (2 * math.pi)) ** 2
        plain = O.rope_frequencies(8, theta)[2]
        assert abs(O.rope_frequencies(8, theta, (4, 1, 4, 1000))[2] / plain - ratio) <= 1e-12, lw
    # every frequency stretched (L tiny): the rotation at position p equals
    # the unscaled one at p / factor; every frequency kept (L huge): unscaled
    x = np.arange(1.0, 17.0).reshape(2, 8)
    assert np.allclose(O.rope(x, 8, 1e4, (4, 1, 4, 1e-3)), O.rope(x, 2, 1e4), atol=1e-13)
    assert np.array_equal(O.rope(x, 8, 1e4, (4, 1, 4, 1e12)), O.rope(x, 8, 1e4))
    # the decode step threads the rule through: a one-layer step whose cached
    # key is the projection rotated with the scaled frequencies
    model_scaled = _rope_probe_model((4, 1, 4, 1e-3))
    model_plain = _rope_probe_model(None)
    kc = [np.zeros((1, 1, 16, 8)) for _ in range(2)]
    vc = [np.zeros((1, 1, 16, 8)) for _ in range(2)]
    O.decode_step(model_scaled, 1, 8, kc[0], vc[0])
    O.decode_step(model_plain, 1, 2, kc[1], vc[1])
    assert np.allclose(kc[0][0, 0, 8], kc[1][0, 0, 2], atol=1e-3)     # fp16 rows of the same rotation
    assert not np.allclose(kc[0][0, 0, 8], O.f16(O.rope(model_plain["probe_k"][None], 8, 1e4))[0], atol=1e-3)


def _rope_probe_model(scaling):
    """One layer, head_dim 8, one query and one KV head; the key projection
    reads a fixed 8-vector out of the normed embedding."""
    h, d = 8, 8
    emb = np.zeros((4, h)); emb[1] = np.arange(1.0, 9.0)
    wk = np.eye(d)
    z = lambda *sh: np.zeros(sh)
    ly = dict(wq=z(d, h), wk=wk, wv=z(d, h), wo=z(h, d), wg=z(4, h), wu=z(4, h), wd=z(h, 4),
              attn_norm=np.ones(h), ffn_norm=np.ones(h))
    m = dict(emb=emb, layers=[ly], norm=np.ones(h), lm_head=np.zeros((4, h)), hq=1, hkv=1, d=d, eps=1e-6,
             theta=1e4, probe_k=O.rmsnorm(np.arange(1.0, 9.0), np.ones(h), 1e-6))
    if scaling is not None:
        m["rope_scaling"] = scaling
    return m


def _h(v: float) -> float:
    """fp16 round to nearest even of a Python float, via struct."""
    return _half_value_struct(_half_bits_struct(v))


def _rms(v, g, eps):
    r = math.sqrt(sum(t * t for t in v) / len(v) + eps)
    return [t / r * w for t, w in zip(v, g)]


def _one_layer(h, d, inter, vocab, **w):
    z = lambda *sh: np.zeros(sh)
    ly = dict(wq=z(d, h), wk=z(d, h), wv=z(d, h), wo=z(h, d), wg=z(inter, h), wu=z(inter, h), wd=z(h, inter),
              attn_norm=np.ones(h), ffn_norm=np.ones(h))
    ly.update({k: np.asarray(v, dtype=np.float64) for k, v in w.items()})
    return ly


def test_decode_step_output_projection_and_ffn_half_closed_form():
    """One layer with zero q/k projections, so position 0 attends to its own
    value row only, and small exact matrices, so each stage has a value
    written out by hand:
      x0 = emb = (1, 1, 1, 1); eps = 0, so h = f16(rmsnorm(x0)) = attn gains
      g_a = (1, 2, 0.5, 1);  v = Wv h = (1, 1, 1, -1) = attention output a;
      x1 = x0 + Wo a = (1.25, 1.5, 1, 1.75)         (the o-projection residual);
      h2 = f16(x1 / rms(x1) * g_f), g_f = (2, 1, 1, 0.5)   (the FFN norm);
      gate = (h2_0, h2_3), up = (h2_1, h2_2);  s = f16(silu(gate) * up)
      (SiLU on the gate branch);  x2 = x1 + Wd s = x1 + (s_0, 0, s_1, 0);
      logits = f16(rmsnorm(x2) * g_n) with an identity LM head.
    A dropped residual, swapped norms, SiLU on the up branch or a transposed
    W_d changes the logits by far more than the fp16 rounding tolerance."""
    g_a, g_f, g_n = [1.0, 2.0, 0.5, 1.0], [2.0, 1.0, 1.0, 0.5], [1.0, 0.5, 2.0, 1.0]
    wv = np.diag([1.0, 0.5, 2.0, -1.0])
    wo = np.diag([0.25, 0.5, 0.0, -0.75])
    wg = np.array([[1.0, 0, 0, 0], [0, 0, 0, 1.0]])
    wu = np.array([[0, 1.0, 0, 0], [0, 0, 1.0, 0]])
    wd = np.array([[1.0, 0], [0, 0], [0, 1.0], [0, 0]])
    ly = _one_layer(4, 4, 2, 4, wv=wv, wo=wo, wg=wg, wu=wu, wd=wd, attn_norm=g_a, ffn_norm=g_f)
    model = dict(emb=np.ones((3, 4)), layers=[ly], norm=np.asarray(g_n), lm_head=np.eye(4), hq=1, hkv=1, d=4,
                 eps=0.0, theta=100.0)
    kc, vc = np.zeros((1, 1, 2, 4)), np.zeros((1, 1, 2, 4))
    logits = O.decode_step(model, 2, 0, kc, vc)

    x1 = [1.25, 1.5, 1.0, 1.75]
    h2 = [_h(t) for t in _rms(x1, g_f, 0.0)]
    gate, up = (h2[0], h2[3]), (h2[1], h2[2])
    s = [_h(g / (1.0 + math.exp(-g)) * u) for g, u in zip(gate, up)]
    x2 = [x1[0] + s[0], x1[1], x1[2] + s[1], x1[3]]
    want = [_h(t) for t in _rms(x2, g_n, 0.0)]
    assert np.allclose(vc[0, 0, 0], [1.0, 1.0, 1.0, -1.0]) and np.all(kc == 0)
    assert np.allclose(logits, want, rtol=0, atol=1e-12), (logits, want)


def test_decode_step_qk_norm_nonuniform_gains_before_rope():
    """Per-head q/k RMSNorm with non-uniform gains, applied before RoPE, at
    position 1 over a cache whose row 0 the test fills by hand.  Hidden 4,
    one head of D = 4, theta = 100 (angles 1 and 0.1 rad at position 1),
    eps = 0, x0 = (1, 1, 1, 1) so the normed input is the attention gains
    g_a = (1, 1, 1, 1); W_q, W_k, W_v are diagonal, so the raw q, k, v are
    the diagonals.  Expected, by hand:
      k1 = f16(rope(rmsnorm(k_raw) * k_norm, 1)), v1 = v_raw,
      q = f16(rope(rmsnorm(q_raw) * q_norm, 1)),
      p = softmax(0.5 * (q . k0, q . k1)), a = p0 v0 + p1 v1,
      x1 = x0 + a (W_o = I), logits = f16(rmsnorm(x1)) (identity head).
    Norm after RoPE, a dropped q_norm or k_norm, or the two gains swapped
    moves the cached key or the softmax weights."""
    q_raw, k_raw, v_raw = [3.0, -1.0, 2.0, 0.5], [1.0, 2.0, -2.0, 4.0], [0.0, 1.0, 0.0, 0.0]
    qn, kn = [1.0, 0.25, 2.0, 0.5], [0.5, 2.0, 1.0, 0.25]
    ly = _one_layer(4, 4, 1, 4, wq=np.diag(q_raw), wk=np.diag(k_raw), wv=np.diag(v_raw), wo=np.eye(4),
                    q_norm=qn, k_norm=kn)
    model = dict(emb=np.ones((2, 4)), layers=[ly], norm=np.ones(4), lm_head=np.eye(4), hq=1, hkv=1, d=4,
                 eps=0.0, theta=100.0)
    kc, vc = np.zeros((1, 1, 3, 4)), np.zeros((1, 1, 3, 4))
    k0, v0 = [0.5, -1.0, 1.0, 0.25], [1.0, 0.0, 0.0, 0.0]
    kc[0, 0, 0], vc[0, 0, 0] = k0, v0
    logits = O.decode_step(model, 1, 1, kc, vc)

    def rot(v):                      # rotate-half pairs (0, 2) by 1 rad and (1, 3) by 0.1 rad
        c0, s0, c1, s1 = math.cos(1.0), math.sin(1.0), math.cos(0.1), math.sin(0.1)
        return [v[0] * c0 - v[2] * s0, v[1] * c1 - v[3] * s1, v[2] * c0 + v[0] * s0, v[3] * c1 + v[1] * s1]
    k1 = [_h(t) for t in rot(_rms(k_raw, kn, 0.0))]
    q = [_h(t) for t in rot(_rms(q_raw, qn, 0.0))]
    s0 = 0.5 * sum(a * b for a, b in zip(q, k0))
    s1 = 0.5 * sum(a * b for a, b in zip(q, k1))
    p0 = 1.0 / (1.0 + math.exp(s1 - s0))
    a = [_h(p0 * v0[i] + (1.0 - p0) * v_raw[i]) for i in range(4)]
    x1 = [1.0 + t for t in a]
    want = [_h(t) for t in _rms(x1, [1.0] * 4, 0.0)]
    assert np.allclose(kc[0, 0, 1], k1, rtol=0, atol=1e-12) and np.allclose(vc[0, 0, 1], v_raw)
    assert np.allclose(logits, want, rtol=0, atol=1e-12), (logits, want)
    assert 0.05 < p0 < 0.95                          # both keys carry weight
