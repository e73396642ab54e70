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


def _experts(seed, e, hidden, inter):
    gw = inputs.weights_np(seed + 1, (e, inter, hidden))
    uw = inputs.weights_np(seed + 2, (e, inter, hidden))
    dw = inputs.weights_np(seed + 3, (e, hidden, inter))
    dev = lambda w: B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), B.Q4_G32), B.LAYOUT_DEVICE)
    def ora(w):
        qs = [O.quantise(w[i], O.Q4) for i in range(e)]
        return np.stack([O.pack(q, O.Q4) for q, _ in qs]), np.stack([s for _, s in qs])
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


@pytest.mark.parametrize("m", workloads.QWEN3_30B_A3B_MOE["m_sweep"])
def test_moe_full_size_sampled_tokens(m):
    """Qwen3-30B-A3B MoE layer at full size: routing of all m tokens is
    bit-exact; the outputs of sampled tokens match the oracle (each token's
    output depends only on its own experts)."""
    cfg = workloads.QWEN3_30B_A3B_MOE
    e, k, hidden, inter = cfg["experts"], cfg["top_k"], cfg["hidden"], cfg["inter"]
    gw = inputs.weights_dev(inputs.seed_for(4, 0, "gate"), (e, inter, hidden))
    uw = inputs.weights_dev(inputs.seed_for(4, 0, "up"), (e, inter, hidden))
    dw = inputs.weights_dev(inputs.seed_for(4, 0, "down"), (e, hidden, inter))
    dev = lambda w: B.qm_repack(B.qm_quantise(w, B.Q4_G32), B.LAYOUT_DEVICE)
    wg, wu, wd = dev(gw), dev(uw), dev(dw)
    x = inputs.activations_dev(inputs.seed_for(4, m, "x"), (m, hidden))
    logits = inputs.logits_dev(inputs.seed_for(4, m, "logits"), (m, e))
    r = _route_check(logits.cpu().numpy(), k)
    y = B.qmoe_grouped_gemm(wg, wu, wd, x, r).cpu().numpy()
    toks = np.array([0, m // 3, m - 1])
    lg = logits.cpu().numpy()[toks]
    ids, _ = O.moe_route(lg, k)
    used = np.unique(ids)
    remap = {int(ex): i for i, ex in enumerate(used)}
    sub = lambda w: w[torch.from_numpy(used).cuda()].cpu().numpy()
    ora = []
    for w in (sub(gw), sub(uw), sub(dw)):
        qs = [O.quantise(w[i], O.Q4) for i in range(len(used))]
        ora += [np.stack([O.pack(q, O.Q4) for q, _ in qs]), np.stack([s for _, s in qs])]
    # the oracle layer over just the experts these tokens use: logits of the
    # other experts are dropped, which leaves each token's top-k unchanged
    lg_sub = lg[:, used]
    ref, ids_sub, *_ = O.moe_layer(x.cpu().numpy()[toks], lg_sub, k, *ora)
    assert np.array_equal(used[ids_sub], ids)
    assert all(remap[int(a)] == b for a, b in zip(ids.ravel(), ids_sub.ravel()))
    assert rel_err(y[toks], ref) <= MFMA_TOL
