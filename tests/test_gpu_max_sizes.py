"""GPU parity at the largest sizes the boundary accepts in one call: GEMM
and prefill attention at m = 65536, routing and bucketing of 65536 tokens,
the MoE layer at m = 65536, and a 32768-row RoPE/cache append ending at the
last row of a 262144-row cache; and very long or very many weight rows
(GEMV at K = 131072 and at a million rows, GEMM at K = 65536).  Outputs
are compared on sampled rows that
the oracle recomputes one by one (first, last and tile-boundary rows
included); routing and bucketing are compared whole, bit for bit."""

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs
from tests.helpers import MFMA_TOL, rel_err

pytestmark = pytest.mark.gpu

M_MAX = 65536


def _rows(rng, m, extra):
    return np.unique(np.concatenate([rng.choice(m, 40, replace=False), [0, m - 1], extra]))


def test_gemm_at_m_max():
    """qmatmul_gemm at m = 65536 with ragged n and a half-empty last K step."""
    n, k = 200, 96
    w = inputs.weights_np(inputs.seed_for(5, n, "gate", 65536), (n, k))
    x = inputs.activations_np(inputs.seed_for(5, M_MAX, "x"), (M_MAX, k))
    wd = B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), B.Q4_G32), B.LAYOUT_DEVICE)
    y = B.qmatmul_gemm(wd, torch.from_numpy(x).cuda()).cpu().numpy()
    assert np.all(np.isfinite(y))
    rows = _rows(np.random.default_rng(65536), M_MAX, [63, 64, 127, 128, M_MAX - 129, M_MAX - 128, M_MAX - 65])
    q, s = O.quantise(w, O.Q4)
    ref = O.gemm(O.pack(q, O.Q4), s, O.Q4, x[rows])
    assert rel_err(y[rows], ref) <= MFMA_TOL


def test_route_and_bucket_at_m_max():
    """qmoe_route over 65536 tokens (524288 assignments, the bucketing split
    over its largest number of workgroups): ids, counts, offsets and the
    stable permutation bit-exact, gates within 1e-6."""
    e, k = 128, 8
    logits = inputs.logits_np(inputs.seed_for(5, M_MAX, "logits"), (M_MAX, e))
    r = B.qmoe_route(torch.from_numpy(logits).cuda(), k)
    torch.cuda.synchronize()
    ids, gates = O.moe_route(logits, k)
    counts, offsets, srt = O.moe_bucket(ids, e)
    assert np.array_equal(r.ids.cpu().numpy(), ids)
    assert np.abs(r.gates.cpu().numpy() - gates).max() <= 1e-6
    assert np.array_equal(r.counts.cpu().numpy(), counts)
    assert np.array_equal(r.offsets.cpu().numpy(), offsets)
    assert np.array_equal(r.sorted_assign.cpu().numpy()[: ids.size], srt)


def test_moe_layer_at_m_max():
    """qmoe_grouped_gemm at m = 65536 (about 4096 rows per expert, many row
    tiles per expert); sampled tokens against the oracle's layer over just
    those tokens (each token's output depends only on its own experts)."""
    e, k, hidden, inter = 128, 8, 128, 64
    gw = inputs.weights_np(inputs.seed_for(5, 1, "gate"), (e, inter, hidden))
    uw = inputs.weights_np(inputs.seed_for(5, 1, "up"), (e, inter, hidden))
    dw = inputs.weights_np(inputs.seed_for(5, 1, "down"), (e, hidden, inter))
    dev = lambda w: B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), B.Q4_G32), B.LAYOUT_DEVICE)
    x = inputs.activations_np(inputs.seed_for(5, M_MAX, "x", 1), (M_MAX, hidden))
    logits = inputs.logits_np(inputs.seed_for(5, M_MAX, "logits", 1), (M_MAX, e))
    r = B.qmoe_route(torch.from_numpy(logits).cuda(), k)
    y = B.qmoe_grouped_gemm(dev(gw), dev(uw), dev(dw), torch.from_numpy(x).cuda(), r).cpu().numpy()
    assert np.all(np.isfinite(y))
    toks = _rows(np.random.default_rng(65537), M_MAX, [M_MAX // 2, M_MAX - 2])

    def deq(w):
        q, s = O.quantise(w, O.Q4)
        return O.dequantise(O.pack(q, O.Q4), s, O.Q4)
    ref, *_ = O.moe_layer_dequantised(x[toks], logits[toks], k, e, lambda i: (deq(gw[i]), deq(uw[i]), deq(dw[i])))
    per_row = np.abs(y[toks] - ref).max(axis=1) / np.abs(ref).max(axis=1)
    assert per_row.max() <= MFMA_TOL, (per_row.max(), toks[int(per_row.argmax())])


@pytest.mark.parametrize("d", [64, 128])
def test_prefill_attention_at_m_max(d):
    """qattn_prefill over a 65536-row prompt from position 0 (the full key
    split plan, fp32 heads out): sampled rows against the oracle's decode
    attention of that row's query over keys 0 .. row."""
    hq, hkv, scale = 2, 1, 1.0 / np.sqrt(d)
    g = torch.Generator(device="cuda").manual_seed(d)
    k = torch.randn((hkv, M_MAX, d), device="cuda", generator=g).half()
    v = torch.randn((hkv, M_MAX, d), device="cuda", generator=g).half()
    q = torch.randn((hq, M_MAX, d), device="cuda", generator=g).half()
    o = B.qattn_prefill(q, k, v, 0, scale).cpu().numpy()
    assert np.all(np.isfinite(o))
    rows = _rows(np.random.default_rng(d), M_MAX, [127, 128, 8191, 8192, M_MAX - 128])
    kn = k.cpu().numpy().astype(np.float64)
    vn = v.cpu().numpy().astype(np.float64)
    qn = q.cpu().numpy()
    ref = np.stack([O.attention_decode(qn[:, i, :], kn, vn, int(i) + 1, scale) for i in rows], axis=1)
    assert rel_err(o[:, rows, :], ref) <= 2e-3


def test_rope_append_rows_to_the_last_cache_row():
    """qdec_rope_append_rows with m = 32768 rows at p0 = 229376, ending at the
    last row of a 262144-row cache, with and without the (cos, sin) table:
    the same bits either way, and sampled rows against the oracle's rotation."""
    hq, hkv, d, max_len, theta = 2, 1, 64, 262144, 1e6
    m = 32768
    p0 = max_len - m
    rng = np.random.default_rng(32768)
    q = torch.from_numpy(rng.standard_normal((m, hq * d)).astype(np.float32)).cuda()
    k = torch.from_numpy(rng.standard_normal((m, hkv * d)).astype(np.float32)).cuda()
    v = torch.from_numpy(rng.standard_normal((m, hkv * d)).astype(np.float32)).cuda()
    kc1 = torch.zeros((hkv, max_len, d), dtype=torch.float16, device="cuda")
    vc1, kc2, vc2 = torch.zeros_like(kc1), torch.zeros_like(kc1), torch.zeros_like(kc1)
    qo1 = B.qdec_rope_append_rows(q, k, v, p0, theta, kc1, vc1)
    qo2 = B.qdec_rope_append_rows(q, k, v, p0, theta, kc2, vc2, table=B.qdec_rope_table(max_len, d, theta))
    assert torch.equal(qo1, qo2) and torch.equal(kc1, kc2) and torch.equal(vc1, vc2)
    qo = qo1.cpu().numpy()
    kcn = kc1[:, p0:].cpu().numpy()
    assert not kc1[:, :p0].any() and not vc1[:, :p0].any()          # rows before p0 untouched
    qn, kn = q.cpu().numpy(), k.cpu().numpy()
    for r in _rows(rng, m, [m - 2]):
        for got, want in ((qo[:, r], O.f16(O.rope(qn[r].reshape(hq, d), p0 + int(r), theta))),
                          (kcn[:, r], O.f16(O.rope(kn[r].reshape(hkv, d), p0 + int(r), theta)))):
            got = got.astype(np.float64)
            assert np.all(np.abs(got - want) <= 2.0 ** -10 * np.abs(want) + 1e-6 * np.abs(want).max()), r
    assert np.array_equal(vc1[:, p0:].cpu().numpy(), v.cpu().numpy().reshape(m, hkv, d).transpose(1, 0, 2)
                          .astype(np.float16))


@pytest.mark.parametrize("fmt", [(O.Q4, B.Q4_G32), (O.Q8, B.Q8_G32), (O.Q3, B.Q3_G32), (O.BF16, B.BF16)])
@pytest.mark.parametrize("n,k", [(100, 131072), (1_000_003, 64)])
def test_gemv_very_long_rows_and_very_many_rows(fmt, n, k):
    """The decode GEMV with K = 131072 (4096 groups: many passes of every
    lane over its chunks, activations from global memory) and with a
    million rows at K = 64 (15,626 panels, a ragged last one); sampled
    rows against the oracle at the GEMV tier."""
    ofmt, bfmt = fmt
    rng = np.random.default_rng(n + k)
    rows = np.unique(np.concatenate([rng.choice(n, 64, replace=False), [0, 63, 64, n - 1]]))
    w = inputs.weights_np(inputs.seed_for(5, n % 1000, "down", k), (n, k))
    x = inputs.activations_np(inputs.seed_for(5, k, "x", 2), (k,))
    wd = B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), bfmt), B.LAYOUT_DEVICE)
    y = B.qmatmul_gemv(wd, torch.from_numpy(x).cuda()).cpu().numpy()
    assert np.all(np.isfinite(y))
    q, s = O.quantise(w[rows], ofmt)
    ref = O.gemv(O.pack(q, ofmt), s, ofmt, x)
    assert rel_err(y[rows], ref) <= 2e-3


def test_gemm_very_long_rows():
    """qmatmul_gemm with K = 65536 at m = 3 (a long split-K), all outputs."""
    m, n, k = 3, 200, 65536
    w = inputs.weights_np(inputs.seed_for(5, n, "up", k), (n, k))
    x = inputs.activations_np(inputs.seed_for(5, m, "x", 3), (m, k))
    wd = B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), B.Q4_G32), B.LAYOUT_DEVICE)
    y = B.qmatmul_gemm(wd, torch.from_numpy(x).cuda()).cpu().numpy()
    q, s = O.quantise(w, O.Q4)
    assert rel_err(y, O.gemm(O.pack(q, O.Q4), s, O.Q4, x)) <= MFMA_TOL
