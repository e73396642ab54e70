"""GPU parity of the weight-format kernels: qm_quantise, qm_dequantise and
qm_repack must be bit-exact with the oracle and with the device layout's
definition."""

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs
from tests.helpers import device_layout

pytestmark = pytest.mark.gpu

FMTS = [(O.Q4, B.Q4_G32), (O.Q8, B.Q8_G32)]


def _gpu_quantise(w_np, fmt):
    w = torch.from_numpy(np.ascontiguousarray(w_np)).cuda()
    qw = B.qm_quantise(w, fmt)
    torch.cuda.synchronize()
    return qw


def _codes(qw):
    return qw.qdata.cpu().numpy(), qw.scales.cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
@pytest.mark.parametrize("n,k", [(1, 32), (3, 96), (65, 64), (130, 1024), (257, 3072)])
def test_quantise_bit_exact(ofmt, bfmt, n, k):
    w = inputs.weights_np(inputs.seed_for(0, n, "q"), (n, k))
    qw = _gpu_quantise(w, bfmt)
    qb, sb = _codes(qw)
    q_ref, s_ref = O.quantise(w, ofmt)
    assert np.array_equal(sb[: n * (k // 32)].reshape(n, k // 32), s_ref)
    assert np.array_equal(qb.reshape(n, -1), O.pack(q_ref, ofmt))


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
def test_quantise_edge_groups_bit_exact(ofmt, bfmt):
    """Ties, one-hot, all-zero, fp16-subnormal scales (the only place Q4's
    -8 appears), tiny groups whose scale underflows to zero, large values."""
    rows = []
    def group(vals):
        g = np.zeros(32, np.float32)
        g[:len(vals)] = vals
        return g
    rows.append(np.concatenate([group([7, -7, 2.5, 3.5, -2.5, -0.5, 0.5, 1.5]), group([0.03])]))
    rows.append(np.concatenate([group([1e-6, -5e-7]), group([-1e-6, 5e-7])]))
    rows.append(np.concatenate([group([]), group([1e-9, -3e-9])]))              # zero, underflow
    rows.append(np.concatenate([group([1000.0, -999.0, 0.1]), group([-127.0, 63.5, 64.5])]))
    rng = np.random.default_rng(5)
    rows.append((rng.standard_normal(64) * 1e-5).astype(np.float32))           # subnormal-scale mix
    w = np.stack(rows).astype(np.float32)
    qw = _gpu_quantise(w, bfmt)
    qb, sb = _codes(qw)
    q_ref, s_ref = O.quantise(w, ofmt)
    assert np.array_equal(sb.reshape(w.shape[0], 2), s_ref)
    assert np.array_equal(qb.reshape(w.shape[0], -1), O.pack(q_ref, ofmt))
    if ofmt == O.Q4:
        assert (q_ref == -8).any()          # the edge really was exercised


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
@pytest.mark.parametrize("batch,n,k", [(1, 1, 32), (1, 65, 96), (3, 70, 64), (1, 200, 2048)])
def test_repack_and_dequantise_bit_exact(ofmt, bfmt, batch, n, k):
    w = inputs.weights_np(inputs.seed_for(0, n + batch, "up"), (batch, n, k))
    qc = _gpu_quantise(w, bfmt)
    qd = B.qm_repack(qc, B.LAYOUT_DEVICE)
    back = B.qm_repack(qd, B.LAYOUT_CANONICAL)
    dq_c = B.qm_dequantise(qc)
    dq_d = B.qm_dequantise(qd)
    torch.cuda.synchronize()
    qdb, qds = _codes(qd)
    per_q = qdb.size // batch
    per_s = qds.size // batch
    for b in range(batch):
        q_ref, s_ref = O.quantise(w[b], ofmt)
        want_q, want_s = device_layout(q_ref, s_ref, ofmt)
        assert np.array_equal(qdb[b * per_q:(b + 1) * per_q], want_q)
        assert np.array_equal(qds[b * per_s:(b + 1) * per_s], want_s)
        ref = O.dequantise(O.pack(q_ref, ofmt), s_ref, ofmt)
        assert np.array_equal(dq_c[b].cpu().numpy().view(np.uint32), ref.view(np.uint32))
        assert np.array_equal(dq_d[b].cpu().numpy().view(np.uint32), ref.view(np.uint32))
    assert torch.equal(back.qdata, qc.qdata) and torch.equal(back.scales, qc.scales)


def test_full_size_lm_head_quantise_sampled_rows():
    """Qwen3-0.6B lm_head (151936 x 1024): GPU codes of sampled rows equal the
    oracle's quantisation of the same fp32 rows."""
    n, k = 151936, 1024
    w = inputs.weights_dev(inputs.seed_for(1, 28, "lm_head"), (n, k))
    qw = B.qm_quantise(w, B.Q4_G32)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, n, 4999), [n - 1]]))
    rows_t = torch.from_numpy(rows).cuda()
    w_rows = w[rows_t].cpu().numpy()
    q_ref, s_ref = O.quantise(w_rows, O.Q4)
    got_q = qw.qdata.view(n, k // 2)[rows_t].cpu().numpy()
    got_s = qw.scales.view(n, k // 32)[rows_t].cpu().numpy().view(np.uint16)
    assert np.array_equal(got_q, O.pack(q_ref, O.Q4))
    assert np.array_equal(got_s, s_ref)
