"""CPU oracle for the weight-only-quantised matrix product (TEST INFRASTRUCTURE).

This module is the correctness reference for the GPU library.  Only the test
suite, the package smoke check and the benchmark's CPU-baseline leg may import
it; the product path never does, and this file imports nothing from the
product package.  Everything here is a plain, slow, deliberately unoptimised
restatement of the definitions, in numpy:

* arithmetic that the method defines in a fixed precision (the group scale,
  the quantised codes) is done in that precision: IEEE fp32 with correctly
  rounded division, round-half-to-even, fp32 -> fp16 round-to-nearest-even;
* every dot product and every MoE step is evaluated in fp64 from the exactly
  dequantised weights, with no blocking, fusion or reordering.

What the method computes comes from the paper's description of its matmul
kernels (Sec. 3.3, "Kernel Fusion and Specialisation": GEMV for M=1 and GEMM
for M>1 per quantisation format, dequantisation integrated into the inner
loop, never materialising dequantised weights; Sec. 3.4, "Prefill": tiled
GEMM for the prompt; Sec. 4.1: the Q4 and Q8 formats and the MoE models).  The
paper states no formula for the format, the routing or the expert FFN; the
group-32 symmetric format, the top-8-then-softmax router and the SwiGLU
experts follow the benchmark workload definitions, and each point the paper
leaves open is resolved as listed in the module docstrings below (the same
readings are collected in the design notes).  The paper names eight weight
formats (Sec. 4.1: Q2, Q3, Q4, Q5, Q6, Q8, BF16, FP16) without defining their
encodings; Q2/Q3/Q5/Q6 here follow the same group-32 symmetric rule as Q4
with qmax = 2^(b-1) - 1, and BF16/FP16 are plain round-to-nearest-even
conversions of the weights.

Pins: every function here is checked by ``tests/test_oracle_pins.py`` against
values fixed by something other than this file (hand-derived IEEE bit
patterns, exact rational arithmetic, integer grids with closed-form answers,
dense-vs-sparse equivalences, brute-force sorting).  The decode-step pieces
are pinned by hand-worked cases: the RoPE angle of every pair against
cos/sin of p * 10^-i (D = 8, theta = 10^4), a one-layer step whose output
projection residual, FFN norm and SwiGLU branch each have a written-out
value, and per-head q/k norms with non-uniform gains checked before RoPE
through the cached key and the softmax weights, and the Llama 3 frequency
rule by its two outer regimes, the linear blend across its band (edges and
midpoint) and the position-scaling identity when every frequency is
stretched.  Each of these fails when the schedule, the residuals, the norm
order, the SiLU branch or a branch of the frequency rule is changed.
"""

from __future__ import annotations

import numpy as np

GROUP = 32
Q4, Q8, Q2, Q3, Q5, Q6, F16, BF16 = 1, 2, 3, 4, 5, 6, 7, 8    # format ids (same numbering as the C ABI)
BITS = {Q2: 2, Q3: 3, Q4: 4, Q5: 5, Q6: 6, Q8: 8}             # integer formats
FLOATS = (F16, BF16)
QMAX = {f: (1 << (b - 1)) - 1 for f, b in BITS.items()}        # Q2 1, Q3 3, Q4 7, Q5 15, Q6 31, Q8 127
QLO = {f: -(1 << (b - 1)) for f, b in BITS.items()}
QLO[Q8] = -127                                                 # Q8 is symmetric
QHI = dict(QMAX)


# ---------------------------------------------------------------------------
# Format: quantise / pack / unpack / dequantise   (Sec. 4.1 formats; Sec. 3.3)
# ---------------------------------------------------------------------------

def fp16_bits(x32: np.ndarray) -> np.ndarray:
    """fp32 -> fp16 bit pattern, round-to-nearest-even (subnormals kept)."""
    return np.asarray(x32, dtype=np.float32).astype(np.float16).view(np.uint16)


def fp16_value(bits: np.ndarray) -> np.ndarray:
    """fp16 bit pattern -> its exact value as fp32."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern, round-to-nearest-even (finite inputs): the
    upper 16 bits of the fp32 pattern, rounded on the lower 16."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    keep = u >> 16
    rest = u & 0xFFFF
    up = (rest > 0x8000) | ((rest == 0x8000) & (keep & 1 == 1))
    return (keep + up).astype(np.uint16)


def bf16_value(bits: np.ndarray) -> np.ndarray:
    """bf16 bit pattern -> its exact value as fp32 (the pattern in the upper
    half of an fp32)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def quantise(w: np.ndarray, fmt: int):
    """Symmetric group-32 quantisation of one weight matrix along K.

    For every row n and every group g of 32 consecutive k:
      m   = max |w|                          (exact, fp32)
      s32 = m / qmax                         (fp32, correctly rounded)
      s16 = fp16_RNE(s32),  s = value(s16)
      q   = 0 everywhere if s == 0, else clamp(rint_half_even(w / s), lo, hi)
    with qmax = 2^(b-1) - 1 and [lo, hi] = [-2^(b-1), 2^(b-1) - 1] for the
    b-bit formats (Q4: 7 and [-8, 7]), except Q8: qmax = 127,
    [lo, hi] = [-127, 127].  The divisor is the fp16-rounded scale, so
    dequantisation lands within s/2 of w and re-quantising is idempotent.

    Returns (q int8 [N][K], s16 uint16 [N][K/32]).  F16 / BF16: returns
    (bits uint16 [N][K], None), each weight rounded to nearest even.
    """
    w = np.asarray(w, dtype=np.float32)
    if w.ndim != 2 or w.shape[1] % GROUP:
        raise ValueError("w must be [N][K] with K a multiple of 32")
    if not np.all(np.isfinite(w)):
        raise ValueError("non-finite weights are outside the format's contract")
    if fmt == F16:
        if np.any(np.abs(w) >= np.float32(65520.0)):
            raise ValueError("weight overflows fp16")
        return fp16_bits(w), None
    if fmt == BF16:
        return bf16_bits(w), None
    n, k = w.shape
    g = w.reshape(n, k // GROUP, GROUP)
    m = np.max(np.abs(g), axis=2)                                  # fp32, exact
    s32 = (m / np.float32(QMAX[fmt])).astype(np.float32)           # IEEE div
    if np.any(s32 > np.float32(65504.0)):
        raise ValueError("group scale overflows fp16")
    s16 = fp16_bits(s32)
    s = fp16_value(s16)
    q = np.zeros((n, k // GROUP, GROUP), dtype=np.float32)
    nz = s != 0
    ratio = np.zeros_like(g)
    ratio[nz] = g[nz] / s[nz][:, None]                             # IEEE div
    q = np.rint(ratio)                                             # half-even
    q = np.clip(q, QLO[fmt], QHI[fmt])
    q[~nz] = 0.0
    return q.reshape(n, k).astype(np.int8), s16.astype(np.uint16)


def pack(q: np.ndarray, fmt: int) -> np.ndarray:
    """Canonical byte packing of the codes of one [N][K] matrix.

    b-bit formats: per row a little-endian bit stream of K*b/8 bytes, code k
    (b-bit two's complement) at bits b*k .. b*k + b - 1, bit i of the stream
    being bit i%8 of byte i/8.  For Q4 that is byte j =
    (q[2j] & 0xF) | ((q[2j+1] & 0xF) << 4); for Q8 the int8 code itself.
    F16 / BF16: the uint16 bit patterns [N][K] unchanged.
    """
    if fmt in FLOATS:
        return np.asarray(q, dtype=np.uint16).copy()
    b = BITS[fmt]
    q = np.asarray(q, dtype=np.int8)
    n, k = q.shape
    u = q.astype(np.int16) & ((1 << b) - 1)                        # two's complement field
    bits = ((u[:, :, None] >> np.arange(b)) & 1).astype(np.uint8)  # [N][K][b], LSB first
    return np.packbits(bits.reshape(n, k * b), axis=1, bitorder="little")


def unpack(qbytes: np.ndarray, fmt: int) -> np.ndarray:
    """Inverse of ``pack``: canonical bytes -> int8 codes [N][K] (F16/BF16:
    the uint16 patterns)."""
    if fmt in FLOATS:
        return np.asarray(qbytes, dtype=np.uint16).copy()
    b = BITS[fmt]
    qb = np.asarray(qbytes, dtype=np.uint8)
    n, nbytes = qb.shape
    k = nbytes * 8 // b
    bits = np.unpackbits(qb, axis=1, bitorder="little").reshape(n, k, b).astype(np.int16)
    u = (bits << np.arange(b)).sum(axis=2)
    return np.where(u >= (1 << (b - 1)), u - (1 << b), u).astype(np.int8)


def dequantise(qbytes: np.ndarray, s16: np.ndarray, fmt: int) -> np.ndarray:
    """w'[n][k] = value(s16[n][k/32]) * q[n][k] as fp32.

    The product of an 11-bit fp16 significand and an integer of at most
    8 bits fits in fp32's 24-bit significand, so this fp32 value is exact.
    F16 / BF16: the value of the stored pattern (exact in fp32).
    """
    if fmt == F16:
        return fp16_value(qbytes)
    if fmt == BF16:
        return bf16_value(qbytes)
    q = unpack(qbytes, fmt).astype(np.float32)
    s = fp16_value(s16)
    n, k = q.shape
    return (q.reshape(n, k // GROUP, GROUP) * s[:, :, None]).reshape(n, k)


def dequantise_f16_tile_value(qbytes: np.ndarray, s16: np.ndarray, fmt: int) -> np.ndarray:
    """The fp16 operand value fp16_RNE(s * q) a half-precision matrix unit
    consumes for one weight (bit pattern, uint16 [N][K]).  This rounding is
    one step more than ``dequantise`` (7 * fp16(0.04/7) is not an fp16).
    F16: the stored pattern itself; BF16: its value rounded to fp16."""
    return fp16_bits(dequantise(qbytes, s16, fmt))


# ---------------------------------------------------------------------------
# GEMV (decode, M = 1) and GEMM (prefill, M > 1)        (Sec. 3.3, Sec. 3.4)
# ---------------------------------------------------------------------------

def gemv(qbytes, s16, fmt, x_f16) -> np.ndarray:
    """y[n] = sum_k w'[n][k] * x[k], evaluated in fp64 (fp64 result [N])."""
    w = dequantise(qbytes, s16, fmt).astype(np.float64)
    x = np.asarray(x_f16, dtype=np.float16).astype(np.float64)
    if x.shape != (w.shape[1],):
        raise ValueError("x must have K entries")
    return w @ x


def gemv_swiglu(gq, gs16, uq, us16, fmt, x_f16) -> np.ndarray:
    """h[n] = silu((Wg' x)[n]) * (Wu' x)[n]: the SwiGLU front half of a
    feed-forward block at batch 1 (Sec. 3.3: fusing the activation into the
    producing kernel), fp64."""
    return silu(gemv(gq, gs16, fmt, x_f16)) * gemv(uq, us16, fmt, x_f16)


def gemm(qbytes, s16, fmt, x_f16) -> np.ndarray:
    """Y[m][n] = sum_k X[m][k] * w'[n][k], in fp64 (fp64 result [M][N])."""
    w = dequantise(qbytes, s16, fmt).astype(np.float64)
    x = np.asarray(x_f16, dtype=np.float16).astype(np.float64)
    if x.ndim != 2 or x.shape[1] != w.shape[1]:
        raise ValueError("X must be [M][K]")
    return x @ w.T


# ---------------------------------------------------------------------------
# Mixture of experts                          (Sec. 4.1 MoE models; Sec. 3.3)
# ---------------------------------------------------------------------------

def moe_route(logits: np.ndarray, top_k: int):
    """Top-k routing of each token.

    For token t the (logit, e) pairs are ordered by logit descending, equal
    logits by lower expert index first; the first top_k experts are kept in
    that order.  The gates are the softmax over just those top_k logits,
    evaluated in fp64 relative to the largest one.

    Returns (ids int32 [M][top_k], gates float64 [M][top_k]).
    """
    lg = np.asarray(logits, dtype=np.float32)
    m, e = lg.shape
    if not 1 <= top_k <= e:
        raise ValueError("need 1 <= top_k <= n_experts")
    ids = np.empty((m, top_k), dtype=np.int32)
    gates = np.empty((m, top_k), dtype=np.float64)
    for t in range(m):
        order = sorted(range(e), key=lambda j: (-float(lg[t, j]), j))[:top_k]
        ids[t] = order
        sel = lg[t, order].astype(np.float64)
        ex = np.exp(sel - sel[0])
        gates[t] = ex / ex.sum()
    return ids, gates


def moe_bucket(ids: np.ndarray, n_experts: int):
    """Counting sort of the M*top_k (token, slot) assignments by expert.

    The flat id of assignment (t, j) is a = t*top_k + j.
      counts[e]   = number of assignments routed to e
      offsets     = exclusive prefix sum of counts, offsets[E] = M*top_k
      sorted_assign lists the flat ids grouped by expert, stably, i.e. in
      ascending a inside each expert.
    Returns (counts int32 [E], offsets int32 [E+1], sorted_assign int32 [M*top_k]).
    """
    flat = np.asarray(ids, dtype=np.int64).reshape(-1)
    counts = np.zeros(n_experts, dtype=np.int64)
    for e in flat:
        counts[e] += 1
    offsets = np.zeros(n_experts + 1, dtype=np.int64)
    for e in range(n_experts):
        offsets[e + 1] = offsets[e] + counts[e]
    cursor = offsets[:-1].copy()
    sorted_assign = np.empty(flat.size, dtype=np.int64)
    for a, e in enumerate(flat):
        sorted_assign[cursor[e]] = a
        cursor[e] += 1
    return counts.astype(np.int32), offsets.astype(np.int32), sorted_assign.astype(np.int32)


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z / (1 + exp(-z)), fp64."""
    return z / (1.0 + np.exp(-z))


def expert_ffn(x64: np.ndarray, wg: np.ndarray, wu: np.ndarray, wd: np.ndarray) -> np.ndarray:
    """SwiGLU expert with no biases, all fp64:
    a = Wg x, b = Wu x, h = silu(a) * b, y = Wd h.  Rows of x64 are tokens."""
    a = x64 @ wg.T
    b = x64 @ wu.T
    h = silu(a) * b
    return h @ wd.T


def dequantise_experts(qbytes, s16, fmt) -> np.ndarray:
    """Stacked experts [E][N][K...] -> fp64 [E][N][K] (exact values)."""
    return np.stack([dequantise(qbytes[e], s16[e], fmt) for e in range(qbytes.shape[0])]).astype(np.float64)


def moe_layer(x_f16, logits, top_k,
              gate_q, gate_s, up_q, up_s, down_q, down_s, fmt=Q4):
    """Routed MoE layer: out[t] = sum_j gates[t][j] * FFN_{ids[t][j]}(x_t),
    with expert e's weights dequantised from its codes and scales.
    Returns (out fp64 [M][H], ids, gates, counts, offsets, sorted_assign).
    """
    def weights(e):
        return (dequantise(gate_q[e], gate_s[e], fmt), dequantise(up_q[e], up_s[e], fmt),
                dequantise(down_q[e], down_s[e], fmt))
    return moe_layer_dequantised(x_f16, logits, top_k, gate_q.shape[0], weights)


def moe_layer_dequantised(x_f16, logits, top_k, n_experts, expert_weights):
    """The routed MoE layer given the dequantised experts:
    expert_weights(e) -> (W'_gate [I][H], W'_up [I][H], W'_down [H][I]).

    Each expert's FFN is applied to the tokens that the bucketing hands it;
    the weighted sum then runs over the slots of each token in slot order.
    Returns (out fp64 [M][H], ids, gates, counts, offsets, sorted_assign).
    """
    x = np.asarray(x_f16, dtype=np.float16).astype(np.float64)
    m = x.shape[0]
    ids, gates = moe_route(logits, top_k)
    counts, offsets, sorted_assign = moe_bucket(ids, n_experts)
    y_assign = None
    for e in range(n_experts):
        rows = sorted_assign[offsets[e]:offsets[e + 1]]
        if rows.size == 0:
            continue
        tok = rows // top_k
        wg, wu, wd = (np.asarray(w, dtype=np.float64) for w in expert_weights(e))
        if y_assign is None:
            y_assign = np.zeros((m * top_k, wd.shape[0]), dtype=np.float64)
        y_assign[rows] = expert_ffn(x[tok], wg, wu, wd)
    if y_assign is None:                       # no tokens
        y_assign = np.zeros((0, np.shape(expert_weights(0)[2])[0]), dtype=np.float64)
    out = np.zeros((m, y_assign.shape[1]), dtype=np.float64)
    for j in range(top_k):
        out += gates[:, j:j + 1] * y_assign[np.arange(m) * top_k + j]
    return out, ids, gates, counts, offsets, sorted_assign


# ---------------------------------------------------------------------------
# Attention over a KV cache                 (Sec. 3.2 KV cache; Sec. 3.4)
# ---------------------------------------------------------------------------

def attention_decode(q, k_cache, v_cache, length: int, scale: float) -> np.ndarray:
    """One decode step of grouped-query attention, in fp64.

    q: [Hq][D]; k_cache, v_cache: [Hkv][Tmax][D], rows t < length valid
    (the cache is sized for the longest context up front, Sec. 3.2).  Query
    head h reads KV head h // (Hq / Hkv).  For each head:
      s_t = scale * (q_h . k_t),  p = softmax(s) over t < length,
      o_h = sum_t p_t v_t.
    Returns o [Hq][D] (fp64).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k_cache, dtype=np.float64)
    v = np.asarray(v_cache, dtype=np.float64)
    hq, d = q.shape
    hkv = k.shape[0]
    if hq % hkv or k.shape != v.shape or k.shape[2] != d or not 1 <= length <= k.shape[1]:
        raise ValueError("bad attention shapes")
    group = hq // hkv
    out = np.empty((hq, d))
    for h in range(hq):
        kk = k[h // group, :length]
        vv = v[h // group, :length]
        sc = scale * (kk @ q[h])
        p = np.exp(sc - sc.max())
        out[h] = (p / p.sum()) @ vv
    return out


def attention_prefill(q, k, v, scale: float, p0: int = 0) -> np.ndarray:
    """Causal grouped-query attention over a prompt chunk, in fp64.

    q: [Hq][M][D], the queries at positions p0 .. p0 + M - 1 (a chunk of a
    prompt processed in bounded chunks, Sec. 3.4); k, v: [Hkv][>= p0 + M][D],
    the keys and values of positions 0 .. p0 + M - 1.  Query row i of head h
    attends to positions j <= p0 + i of KV head h // (Hq / Hkv) with
    softmax(scale * q_i . k_j).  Returns o [Hq][M][D] (fp64).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    hq, m, d = q.shape
    hkv = k.shape[0]
    n = p0 + m
    if hq % hkv or k.shape[0] != hkv or k.shape[1] < n or k.shape[2] != d or v.shape != k.shape:
        raise ValueError("bad attention shapes")
    group = hq // hkv
    out = np.empty((hq, m, d))
    mask = np.arange(n)[None, :] <= (p0 + np.arange(m))[:, None]     # [M][n]
    for h in range(hq):
        sc = scale * (q[h] @ k[h // group, :n].T)                     # [M][n]
        sc = np.where(mask, sc, -np.inf)
        p = np.exp(sc - sc.max(axis=1, keepdims=True))
        out[h] = (p / p.sum(axis=1, keepdims=True)) @ v[h // group, :n]
    return out


# ---------------------------------------------------------------------------
# One decode step of a dense decoder             (Sec. 3.2, Sec. 3.3)
# ---------------------------------------------------------------------------

def rmsnorm(x, w, eps: float) -> np.ndarray:
    """y = x / sqrt(mean(x^2) + eps) * w, fp64."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x) + eps) * np.asarray(w, dtype=np.float64)


def rope_frequencies(d: int, theta: float, scaling=None) -> np.ndarray:
    """Rotation frequency of each pair i < D/2, fp64: theta^(-2i/D).

    scaling = (factor, low_freq_factor, high_freq_factor, original_len)
    applies the Llama 3 family's long-context rule to each frequency f with
    wavelength w = 2 pi / f, taking L = original_len:
      w < L / high_freq_factor  -> f (short wavelengths kept),
      w > L / low_freq_factor   -> f / factor (long wavelengths stretched),
      otherwise                 -> (1 - t) f / factor + t f,
                                   t = (L / w - low_freq_factor) / (high_freq_factor - low_freq_factor),
    so the middle band blends linearly in L / w between the two outer rules
    (t = 0 and t = 1 at its edges).  The paper runs Llama 3.2 models without
    stating their RoPE; this is the rule those models are published with."""
    i = np.arange(d // 2)
    f = float(theta) ** (-2.0 * i / d)
    if scaling is None:
        return f
    factor, lo, hi, orig = (float(v) for v in scaling)
    w = 2.0 * np.pi / f
    t = (orig / w - lo) / (hi - lo)
    mid = (1.0 - t) * f / factor + t * f
    return np.where(w < orig / hi, f, np.where(w > orig / lo, f / factor, mid))


def rope(x, pos: int, theta: float, scaling=None) -> np.ndarray:
    """Rotary position embedding of each head row of x [H][D] at position
    pos, pairing dimension i with i + D/2 (the Llama / Qwen convention):
    angle_i = pos * f_i with f_i from rope_frequencies (theta^(-2i/D) when
    unscaled), (a, b) -> (a cos - b sin, b cos + a sin)."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    ang = pos * rope_frequencies(d, theta, scaling)
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :d // 2], x[..., d // 2:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def f16(x) -> np.ndarray:
    """Round to fp16 (the precision of every activation a kernel hands to
    the next one) and return the value as fp64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float16).astype(np.float64)


def greedy_token(logits) -> int:
    """Greedy sampling: the first index of the largest non-NaN logit (0 when
    every logit is NaN)."""
    z = np.asarray(logits, dtype=np.float64)
    ok = ~np.isnan(z)
    if not ok.any():
        return 0
    return int(np.flatnonzero(ok & (z == z[ok].max()))[0])


def decode_step(model: dict, token: int, pos: int, k_cache: np.ndarray, v_cache: np.ndarray) -> np.ndarray:
    """Logits of one decode step of a dense grouped-query-attention decoder
    with SwiGLU feed-forward blocks (the Llama 3.2 / Qwen3 layer), in fp64.

    model: emb [V][H] and the norm weights as fp16 values; per layer the
    dequantised projections wq, wk, wv, wo, wg, wu, wd ([N][K], fp64) and
    attn_norm, ffn_norm; norm, lm_head; hq, hkv, d, eps, theta.  The
    activations handed between kernels are rounded to fp16 where the kernels'
    interfaces are fp16: the normed inputs of every projection, q after
    RoPE, the new K / V rows (written into k_cache / v_cache [L][Hkv][T][D]
    at row pos), the attention output and the SwiGLU output.  The residual
    stream stays fp32 on the GPU and fp64 here.  A layer with "q_norm" and
    "k_norm" gains ([D], the Qwen3 layer) RMS-normalises every query and key
    head over its D dimensions before RoPE.  An optional "rope_scaling"
    (factor, low_freq_factor, high_freq_factor, original_len) selects the
    Llama 3 frequency rule of rope_frequencies.
    """
    hq, hkv, d, eps, theta = model["hq"], model["hkv"], model["d"], model["eps"], model["theta"]
    scaling = model.get("rope_scaling")
    x = np.asarray(model["emb"][token], dtype=np.float64)
    for li, ly in enumerate(model["layers"]):
        h = f16(rmsnorm(x, ly["attn_norm"], eps))
        q = (ly["wq"] @ h).reshape(hq, d)
        k = (ly["wk"] @ h).reshape(hkv, d)
        if "q_norm" in ly:
            q = np.stack([rmsnorm(r, ly["q_norm"], eps) for r in q])
            k = np.stack([rmsnorm(r, ly["k_norm"], eps) for r in k])
        q = rope(q, pos, theta, scaling)
        k = rope(k, pos, theta, scaling)
        v = (ly["wv"] @ h).reshape(hkv, d)
        k_cache[li, :, pos] = f16(k)
        v_cache[li, :, pos] = f16(v)
        a = attention_decode(f16(q), k_cache[li], v_cache[li], pos + 1, 1.0 / np.sqrt(d))
        x = x + ly["wo"] @ f16(a.reshape(-1))
        h = f16(rmsnorm(x, ly["ffn_norm"], eps))
        x = x + ly["wd"] @ f16(silu(ly["wg"] @ h) * (ly["wu"] @ h))
    return model["lm_head"] @ f16(rmsnorm(x, model["norm"], eps))
