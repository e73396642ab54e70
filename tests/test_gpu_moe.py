"""GPU parity of the MoE path: routing and bucketing bit-exact, the grouped
expert layer within the fp16-MFMA tolerance."""

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs, workloads
from tests.helpers import MFMA_TOL, rel_err

pytestmark = pytest.mark.gpu


def _route_check(logits, top_k):
    r = B.qmoe_route(torch.from_numpy(logits).cuda(), top_k)
    torch.cuda.synchronize()
    ids, gates = O.moe_route(logits, top_k)
    counts, offsets, srt = O.moe_bucket(ids, logits.shape[1])
    assert np.array_equal(r.ids.cpu().numpy(), ids)
    assert np.abs(r.gates.cpu().numpy() - gates).max() <= 1e-6
    assert np.array_equal(r.counts.cpu().numpy(), counts)
    assert np.array_equal(r.offsets.cpu().numpy(), offsets)
    assert np.array_equal(r.sorted_assign.cpu().numpy()[: ids.size], srt)
    return r


@pytest.mark.parametrize("m,e,k", [(1, 128, 8), (37, 128, 8), (300, 100, 4), (1000, 1024, 16),
                                   (64, 8, 8), (50, 3, 1), (2048, 128, 8),
                                   (256, 128, 8), (257, 128, 8),     # one / two bucketing workgroups
                                   (5000, 64, 8),                    # 16 bucketing workgroups
                                   (120, 256, 16), (90, 200, 6)])    # 4 logits per lane
def test_route_bit_exact(m, e, k):
    logits = inputs.logits_np(inputs.seed_for(4, m, "logits"), (m, e))
    _route_check(logits, k)


def test_route_ties_and_adversarial():
    m, e = 200, 128
    logits = np.zeros((m, e), np.float32)               # all ties: experts 0..7 every token
    _route_check(logits, 8)
    rng = np.random.default_rng(2)
    logits = rng.integers(-2, 3, size=(m, e)).astype(np.float32)   # many ties
    _route_check(logits, 8)
    logits = np.full((m, e), -1.0, np.float32)
    logits[:, 127] = 5.0                                 # one hot expert, others tied
    logits[::2, 0] = -0.0
    _route_check(logits, 8)


def test_bucket_skewed_across_workgroup_slices():
    """All 4096 tokens tie and pick experts 0..7: every expert's 4096
    assignments span all 16 bucketing slices, so each slice's base must count
    the earlier slices exactly."""
    _route_check(np.zeros((4096, 128), np.float32), 8)
    logits = np.zeros((4096, 128), np.float32)
    logits[1::2, 100:108] = 1.0                           # odd tokens: experts 100..107
    _route_check(logits, 8)


def test_route_empty():
    logits = np.zeros((0, 16), np.float32)
    r = B.qmoe_route(torch.zeros((0, 16), device="cuda"), 2)
    torch.cuda.synchronize()
    assert r.counts.cpu().numpy().tolist() == [0] * 16
    assert r.offsets.cpu().numpy().tolist() == [0] * 17
    del logits


def _experts(seed, e, hidden, inter, fmts=(O.Q4, B.Q4_G32)):
    ofmt, bfmt = fmts
    gw = inputs.weights_np(seed + 1, (e, inter, hidden))
    uw = inputs.weights_np(seed + 2, (e, inter, hidden))
    dw = inputs.weights_np(seed + 3, (e, hidden, inter))
    dev = lambda w: B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), bfmt), B.LAYOUT_DEVICE)
    def ora(w):
        qs = [O.quantise(w[i], ofmt) for i in range(e)]
        return np.stack([O.pack(q, ofmt) for q, _ in qs]), np.stack([s for _, s in qs])
    return (dev(gw), dev(uw), dev(dw)), ora(gw) + ora(uw) + ora(dw)


@pytest.mark.parametrize("m,e,k,hidden,inter", [
    (1, 8, 2, 64, 96),          # single token
    (40, 16, 4, 128, 96),       # ragged tiles, some experts empty
    (100, 128, 8, 256, 192),    # many experts, ~6 rows each (small-M tiles)
    (600, 16, 8, 128, 64),      # ~300 rows per expert (large-M tiles)
    (70, 32, 1, 96, 128),       # top-1
])
def test_moe_layer_parity(m, e, k, hidden, inter):
    (wg, wu, wd), ora = _experts(1000 + m, e, hidden, inter)
    x = inputs.activations_np(inputs.seed_for(4, m, "x"), (m, hidden))
    logits = inputs.logits_np(inputs.seed_for(4, m, "logits"), (m, e))
    r = _route_check(logits, k)
    y = B.qmoe_grouped_gemm(wg, wu, wd, torch.from_numpy(x).cuda(), r).cpu().numpy()
    ref, *_ = O.moe_layer(x, logits, k, *ora)
    assert rel_err(y, ref) <= MFMA_TOL


@pytest.mark.parametrize("fmts", [(O.Q2, B.Q2_G32), (O.Q3, B.Q3_G32), (O.Q5, B.Q5_G32), (O.Q6, B.Q6_G32),
                                  (O.Q8, B.Q8_G32)], ids=["q2", "q3", "q5", "q6", "q8"])
@pytest.mark.parametrize("m,e,k,hidden,inter", [
    (40, 16, 4, 128, 96),       # ragged tiles, some experts empty
    (100, 128, 8, 256, 192),    # ~6 rows per expert: 32-row tiles, nontemporal weights
    (200, 32, 8, 128, 96),      # ~50 rows per expert: middle plan
    (600, 16, 8, 128, 64),      # ~300 rows per expert: several row tiles per expert
])
def test_moe_layer_parity_other_formats(fmts, m, e, k, hidden, inter):
    """Experts in Q2/Q3/Q5/Q6/Q8 through every tile plan, against the
    oracle's layer on the same codes and scales."""
    (wg, wu, wd), ora = _experts(2000 + m, e, hidden, inter, fmts)
    x = inputs.activations_np(inputs.seed_for(5, m, "x"), (m, hidden))
    logits = inputs.logits_np(inputs.seed_for(5, m, "logits"), (m, e))
    r = _route_check(logits, k)
    y = B.qmoe_grouped_gemm(wg, wu, wd, torch.from_numpy(x).cuda(), r).cpu().numpy()
    ref, *_ = O.moe_layer(x, logits, k, *ora, fmt=fmts[0])
    assert rel_err(y, ref) <= MFMA_TOL


def test_moe_all_tokens_to_eight_experts_and_determinism():
    m, e, k, hidden, inter = 257, 128, 8, 128, 64
    (wg, wu, wd), ora = _experts(77, e, hidden, inter)
    x = inputs.activations_np(78, (m, hidden))
    logits = np.zeros((m, e), np.float32)
    logits[:, 64:72] = np.arange(8, dtype=np.float32)   # experts 64..71 hot, 120 empty
    r = _route_check(logits, k)
    xt = torch.from_numpy(x).cuda()
    y1 = B.qmoe_grouped_gemm(wg, wu, wd, xt, r)
    y2 = B.qmoe_grouped_gemm(wg, wu, wd, xt, r)
    assert torch.equal(y1, y2)
    ref, *_ = O.moe_layer(x, logits, k, *ora)
    assert rel_err(y1.cpu().numpy(), ref) <= MFMA_TOL


@pytest.fixture(scope="module")
def full_size_experts():
    """The Qwen3-30B-A3B experts (128 x gate/up 2048 -> 768, down 768 ->
    2048, Q4) on the device, and the oracle's dequantised copies of the same
    seeded weights (quantised, packed and dequantised by the oracle, one
    thread per expert matrix)."""
    import concurrent.futures as cf
    cfg = workloads.QWEN3_30B_A3B_MOE
    e, hidden, inter = cfg["experts"], cfg["hidden"], cfg["inter"]
    raw = [inputs.weights_dev(inputs.seed_for(4, 0, t), sh) for t, sh in
           (("gate", (e, inter, hidden)), ("up", (e, inter, hidden)), ("down", (e, hidden, inter)))]
    dev = [B.qm_repack(B.qm_quantise(w, B.Q4_G32), B.LAYOUT_DEVICE) for w in raw]
    host = [w.cpu().numpy() for w in raw]
    del raw

    def deq(w):
        q, sc = O.quantise(w, O.Q4)
        return O.dequantise(O.pack(q, O.Q4), sc, O.Q4)
    with cf.ThreadPoolExecutor(16) as ex:
        ora = [list(ex.map(deq, list(h))) for h in host]
    return dev, ora


def _full_size_tokens(m, ids, rng):
    """All tokens for m <= 128; else 128 or more tokens that hit, in each of
    the three largest experts' buckets, the first, middle and last row of
    every 16-row block (so every row tile of every tile plan), topped up with
    random tokens."""
    if m <= 128:
        return np.arange(m)
    k = ids.shape[1]
    _, _, sorted_assign = O.moe_bucket(ids, int(ids.max()) + 1)
    counts = np.bincount(ids.ravel())
    offsets = np.concatenate([[0], np.cumsum(counts)])
    pick = set()
    for ex in np.argsort(-counts, kind="stable")[:3]:
        bucket = sorted_assign[offsets[ex]:offsets[ex + 1]]
        for b0 in range(0, len(bucket), 16):
            blk = bucket[b0:b0 + 16]
            pick.update(int(a) // k for a in (blk[0], blk[len(blk) // 2], blk[-1]))
    rest = np.setdiff1d(np.arange(m), np.array(sorted(pick)))
    need = max(0, 128 - len(pick))
    pick.update(int(t) for t in rng.choice(rest, size=need, replace=False))
    return np.array(sorted(pick))


@pytest.mark.parametrize("m", workloads.QWEN3_30B_A3B_MOE["m_sweep"])
def test_moe_full_size_sampled_tokens(m, full_size_experts):
    """Qwen3-30B-A3B MoE layer at full size: routing of all m tokens is
    bit-exact; the output rows of all tokens (m = 128) or of at least 128
    tokens that cover every row tile of the three largest buckets match the
    oracle row by row (each token's output depends only on its own
    experts)."""
    cfg = workloads.QWEN3_30B_A3B_MOE
    e, k, hidden = cfg["experts"], cfg["top_k"], cfg["hidden"]
    (wg, wu, wd), ora = full_size_experts
    x = inputs.activations_dev(inputs.seed_for(4, m, "x"), (m, hidden))
    logits = inputs.logits_dev(inputs.seed_for(4, m, "logits"), (m, e))
    lg = logits.cpu().numpy()
    r = _route_check(lg, k)
    y = B.qmoe_grouped_gemm(wg, wu, wd, x, r).cpu().numpy()
    ids_all, _ = O.moe_route(lg, k)
    toks = _full_size_tokens(m, ids_all, np.random.default_rng(m))
    assert len(toks) >= min(m, 128)
    ref, ids, *_ = O.moe_layer_dequantised(x.cpu().numpy()[toks], lg[toks], k, e,
                                           lambda ex: (ora[0][ex], ora[1][ex], ora[2][ex]))
    assert np.array_equal(ids, ids_all[toks])
    got = y[toks]
    assert np.all(np.isfinite(got))
    per_row = np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)
    assert per_row.max() <= MFMA_TOL, (per_row.max(), toks[int(per_row.argmax())])


def test_moe_topk_ids_checked_against_buckets():
    """An assignment whose bucket is not the expert topk_ids names turns its
    token's output row into NaN; every other row is unchanged."""
    m, e, k, hidden, inter = 48, 16, 4, 128, 96
    (wg, wu, wd), _ = _experts(4242, e, hidden, inter)
    x = torch.from_numpy(inputs.activations_np(inputs.seed_for(4, m, "x"), (m, hidden))).cuda()
    logits = inputs.logits_np(inputs.seed_for(4, m, "logits"), (m, e))
    r = _route_check(logits, k)
    y0 = B.qmoe_grouped_gemm(wg, wu, wd, x, r)
    bad = 17                                   # token 17, slot 2: claim another expert
    ids = r.ids.clone()
    ids[bad, 2] = (ids[bad, 2] + 1) % e
    r2 = B.Routing(ids, r.gates, r.counts, r.offsets, r.sorted_assign, r.top_k)
    y1 = B.qmoe_grouped_gemm(wg, wu, wd, x, r2)
    nan_rows = torch.isnan(y1).any(dim=1).cpu().numpy()
    assert nan_rows[bad] and nan_rows.sum() == 1
    keep = torch.ones(m, dtype=torch.bool); keep[bad] = False
    assert torch.equal(y0[keep.cuda()], y1[keep.cuda()])
