"""GPU parity of decode attention over a KV cache (qattn_decode) with the
oracle."""

import math

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from tests.helpers import rel_err

pytestmark = pytest.mark.gpu

ATTN_TOL = 2e-5    # fp32 scores, exp2 and sums against fp64


def _case(hq, hkv, d, length, max_len, seed, scale=None, poison=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((hq, d)).astype(np.float16)
    k = rng.standard_normal((hkv, max_len, d)).astype(np.float16)
    v = rng.standard_normal((hkv, max_len, d)).astype(np.float16)
    if poison and length < max_len:
        # rows past the length are not data: NaN there must not reach o
        k[:, length:] = np.float16(np.nan)
        v[:, length:] = np.float16(np.inf)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    o = B.qattn_decode(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda(),
                       length, scale).cpu().numpy()
    ref = O.attention_decode(q, k[:, :length], v[:, :length], length, np.float32(scale))
    return o, ref


# Group sizes 1-8, head_dim 64 and 128, a single row, ragged slices, lengths
# that need many slices, a full cache.
@pytest.mark.parametrize("hq,hkv,d,length,max_len", [
    (16, 8, 128, 1, 64), (16, 8, 128, 33, 64), (24, 8, 128, 1000, 1024), (32, 8, 64, 4097, 8192),
    (8, 8, 64, 100, 128), (64, 8, 128, 777, 1000), (12, 4, 128, 5000, 5000), (40, 8, 64, 31, 31),
    (14, 2, 128, 20000, 32768), (7, 1, 64, 3, 16)])
def test_attn_decode_parity(hq, hkv, d, length, max_len):
    o, ref = _case(hq, hkv, d, length, max_len, seed=hq * 1000 + length)
    assert np.all(np.isfinite(o))
    assert rel_err(o, ref) <= ATTN_TOL


def test_attn_decode_sharp_softmax():
    """Scale 1 on unit-variance q, k: scores spread over tens, so the slice
    maxima and the cross-slice merge decide the result."""
    o, ref = _case(16, 8, 128, 3000, 4096, seed=7, scale=1.0)
    assert rel_err(o, ref) <= ATTN_TOL


def test_attn_decode_long_context_sampled_heads():
    """Qwen3-0.6B attention shape (16 query heads, 8 KV heads, head_dim 128)
    at the longest supported context, 262144 rows (256 slices of 1024)."""
    hq, hkv, d, length = 16, 8, 128, 262144
    g = torch.Generator(device="cuda").manual_seed(11)
    q = torch.randn((hq, d), generator=g, device="cuda").half()
    k = torch.randn((hkv, length, d), generator=g, device="cuda").half()
    v = torch.randn((hkv, length, d), generator=g, device="cuda").half()
    o = B.qattn_decode(q, k, v, length, 1.0 / math.sqrt(d)).cpu().numpy()
    for kvh in (0, 5):
        ref = O.attention_decode(q[2 * kvh:2 * kvh + 2].cpu().numpy(), k[kvh:kvh + 1].cpu().numpy(),
                                 v[kvh:kvh + 1].cpu().numpy(), length, np.float32(1.0 / math.sqrt(d)))
        assert rel_err(o[2 * kvh:2 * kvh + 2], ref) <= ATTN_TOL


def test_attn_decode_deterministic_and_workspace_reuse():
    rng = np.random.default_rng(3)
    hq, hkv, d, n = 24, 8, 128, 2048
    q = torch.from_numpy(rng.standard_normal((hq, d)).astype(np.float16)).cuda()
    k = torch.from_numpy(rng.standard_normal((hkv, n, d)).astype(np.float16)).cuda()
    v = torch.from_numpy(rng.standard_normal((hkv, n, d)).astype(np.float16)).cuda()
    ws = torch.empty(B.qattn_decode_workspace_bytes(hq, d), dtype=torch.uint8, device="cuda")
    a = B.qattn_decode(q, k, v, n, 0.1, workspace=ws)
    b = B.qattn_decode(q, k, v, 17, 0.1, workspace=ws)          # another length in between
    c = B.qattn_decode(q, k, v, n, 0.1, workspace=ws)
    assert torch.equal(a, c)
    ref = O.attention_decode(q.cpu().numpy(), k.cpu().numpy()[:, :17], v.cpu().numpy()[:, :17], 17, np.float32(0.1))
    assert rel_err(b.cpu().numpy(), ref) <= ATTN_TOL


PREFILL_TOL = 1e-2     # fp16 MFMA operands (p rounded to fp16)


def _prefill_case(hq, hkv, d, m, p0, max_len, seed, scale=None):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((hq, m, d)).astype(np.float16)
    k = rng.standard_normal((hkv, max_len, d)).astype(np.float16)
    v = rng.standard_normal((hkv, max_len, d)).astype(np.float16)
    if p0 + m < max_len:
        k[:, p0 + m:] = np.float16(np.nan)          # positions past the chunk are not data
        v[:, p0 + m:] = np.float16(np.nan)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    o = B.qattn_prefill(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda(),
                        p0, scale).cpu().numpy()
    return o, q, k, v, scale


# Llama-3.2-1B (32 / 8 heads, head_dim 64) and Qwen3 / Llama-3.2-3B style
# (head_dim 128) shapes; ragged chunks, chunks at an offset, one row.
@pytest.mark.parametrize("hq,hkv,d,m,p0,max_len", [
    (4, 2, 64, 1, 0, 8), (4, 2, 128, 33, 0, 40), (8, 8, 64, 200, 0, 256), (6, 2, 128, 300, 0, 300),
    (4, 1, 64, 129, 77, 400), (32, 8, 64, 512, 0, 512), (16, 8, 128, 250, 1000, 1300),
    (24, 8, 128, 128, 0, 128)])
def test_attn_prefill_parity(hq, hkv, d, m, p0, max_len):
    o, q, k, v, scale = _prefill_case(hq, hkv, d, m, p0, max_len, seed=m + p0 + d)
    ref = O.attention_prefill(q, k[:, :p0 + m], v[:, :p0 + m], np.float32(scale), p0=p0)
    assert np.all(np.isfinite(o))
    err = rel_err(o, ref)
    assert err <= PREFILL_TOL
    assert err <= 2e-3, err


def test_attn_prefill_full_prompt_sampled_rows():
    """Llama-3.2-1B attention shape at M = 2048: sampled query rows of
    sampled heads against the oracle, both ends of the causal range."""
    hq, hkv, d, m = 32, 8, 64, 2048
    o, q, k, v, scale = _prefill_case(hq, hkv, d, m, 0, m, seed=99)
    rows = np.array([0, 1, 127, 128, 1000, 2046, 2047])
    for h in (0, 9, 31):
        for i in rows:
            ref = O.attention_decode(q[h:h + 1, i], k[h // 4:h // 4 + 1], v[h // 4:h // 4 + 1], int(i) + 1,
                                     np.float32(scale))
            assert rel_err(o[h, i][None], ref) <= PREFILL_TOL


@pytest.mark.parametrize("hq,hkv,d,m", [(24, 8, 64, 2400), (20, 4, 128, 4000)])
def test_attn_prefill_every_tile_of_every_head(hq, hkv, d, m):
    """Grids of 456 and 640 workgroups: more than one round over the CUs,
    with partial last rounds (the reversed dealing of every second round).
    One sampled query row of every (head, 128-row tile) unit against the
    oracle, so a unit computed twice or never shows up."""
    o, q, k, v, scale = _prefill_case(hq, hkv, d, m, 0, m, seed=m + d)
    assert np.all(np.isfinite(o))
    g = hq // hkv
    for h in range(hq):
        for t in range((m + 127) // 128):
            i = min(m - 1, t * 128 + (37 * h + 11 * t) % 128)
            ref = O.attention_decode(q[h:h + 1, i], k[h // g:h // g + 1], v[h // g:h // g + 1], int(i) + 1,
                                     np.float32(scale))
            assert rel_err(o[h, i][None], ref) <= PREFILL_TOL, (h, t, i)


@pytest.mark.parametrize("hq,hkv,d,m,p0", [(16, 8, 128, 1000, 0), (8, 2, 64, 300, 20000), (12, 4, 128, 700, 300)])
def test_attn_prefill_key_splits(hq, hkv, d, m, p0):
    """Long tiles split over key ranges (full workspace), fewer splits (a
    third of it) and none (no workspace): each against the oracle, each
    repeatable bit for bit."""
    max_len = p0 + m
    rng = np.random.default_rng(m + d)
    q = rng.standard_normal((hq, m, d)).astype(np.float16)
    k = rng.standard_normal((hkv, max_len, d)).astype(np.float16)
    v = rng.standard_normal((hkv, max_len, d)).astype(np.float16)
    scale = 1.0 / math.sqrt(d)
    qd, kd, vd = (torch.from_numpy(a).cuda() for a in (q, k, v))
    need = B.qattn_prefill_workspace_bytes(hq, d, m, p0)
    assert need > 0                                       # these shapes split on a 256-CU part
    ref = O.attention_prefill(q, k, v, np.float32(scale), p0=p0)
    outs = []
    for ws in (torch.empty(need, dtype=torch.uint8, device="cuda"),
               torch.empty(need // 3 // 16 * 16, dtype=torch.uint8, device="cuda"), B.NO_WORKSPACE):
        o1 = B.qattn_prefill(qd, kd, vd, p0, scale, workspace=ws).cpu().numpy()
        o2 = B.qattn_prefill(qd, kd, vd, p0, scale, workspace=ws).cpu().numpy()
        assert np.array_equal(o1, o2)
        assert np.all(np.isfinite(o1))
        assert rel_err(o1, ref) <= PREFILL_TOL
        outs.append(o1)
    # Each split rounds its p to fp16 (toward zero, 2^-10 relative) against
    # its own running maximum, so the plans differ at that rounding: two
    # independent 2^-10 perturbations of the weights of an average.
    assert rel_err(outs[0], outs[2].astype(np.float64)) <= 2.0 ** -9
    assert rel_err(outs[1], outs[2].astype(np.float64)) <= 2.0 ** -9


def test_attn_prefill_chunk_far_into_cache():
    """A 128-row chunk at position 100,000 (one query tile per head, split
    over key ranges): sampled rows against the oracle's decode attention over
    each row's prefix, and the unsplit form within the p rounding."""
    hq, hkv, d, m, p0 = 16, 8, 128, 128, 100_000
    max_len = p0 + m
    g = torch.Generator(device="cuda").manual_seed(7)
    q = torch.randn((hq, m, d), generator=g, device="cuda").half()
    k = torch.randn((hkv, max_len, d), generator=g, device="cuda").half()
    v = torch.randn((hkv, max_len, d), generator=g, device="cuda").half()
    scale = 1.0 / math.sqrt(d)
    assert B.qattn_prefill_workspace_bytes(hq, d, m, p0) > 0
    o = B.qattn_prefill(q, k, v, p0, scale).cpu().numpy()
    o_none = B.qattn_prefill(q, k, v, p0, scale, workspace=B.NO_WORKSPACE).cpu().numpy()
    assert rel_err(o, o_none.astype(np.float64)) <= 2.0 ** -9
    qn, kn, vn = q.cpu().numpy(), k.cpu().numpy(), v.cpu().numpy()
    for h in (0, 7, 15):
        for i in (0, 1, 63, 127):
            ref = O.attention_decode(qn[h:h + 1, i], kn[h // 2:h // 2 + 1], vn[h // 2:h // 2 + 1], p0 + i + 1,
                                     np.float32(scale))
            assert rel_err(o[h, i][None], ref) <= PREFILL_TOL, (h, i)


@pytest.mark.parametrize("hq,hkv,d,m,p0", [(8, 2, 64, 300, 0), (16, 8, 128, 1000, 0), (12, 4, 128, 128, 20000)])
def test_attn_prefill_rows_f16_equals_heads_then_rows(hq, hkv, d, m, p0):
    """The fp16-rows form (unsplit and key-split) equals qattn_prefill followed
    by qdec_heads_to_rows_f16, bit for bit."""
    g = torch.Generator(device="cuda").manual_seed(m + d)
    q = torch.randn((hq, m, d), generator=g, device="cuda").half()
    k = torch.randn((hkv, p0 + m, d), generator=g, device="cuda").half()
    v = torch.randn((hkv, p0 + m, d), generator=g, device="cuda").half()
    scale = 1.0 / math.sqrt(d)
    for ws in (None, B.NO_WORKSPACE):
        o = B.qattn_prefill(q, k, v, p0, scale, workspace=ws)
        want = B.qdec_heads_to_rows_f16(o)
        got = B.qattn_prefill_rows_f16(q, k, v, p0, scale, workspace=ws)
        assert torch.equal(got.view(torch.int16), want.view(torch.int16))


def test_attn_prefill_last_row_matches_decode():
    """The last query of a chunk attends to the whole prefix: it equals the
    decode kernel's result for that query (within the MFMA tolerance)."""
    hq, hkv, d, m, p0 = 16, 8, 128, 96, 160
    o, q, k, v, scale = _prefill_case(hq, hkv, d, m, p0, p0 + m, seed=5)
    dec = B.qattn_decode(torch.from_numpy(np.ascontiguousarray(q[:, -1])).cuda(), torch.from_numpy(k).cuda(),
                         torch.from_numpy(v).cuda(), p0 + m, scale).cpu().numpy()
    assert rel_err(o[:, -1], dec.astype(np.float64)) <= PREFILL_TOL
    o2 = B.qattn_prefill(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda(),
                         p0, scale).cpu().numpy()
    assert np.array_equal(o, o2)                     # deterministic
