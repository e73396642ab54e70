"""Seeded random shapes across every weight format: the GEMV (m = 1), the
MFMA GEMM, the grouped GEMM and the MoE layer against the oracle, on
sampled outputs.  The shapes are drawn log-uniformly (M up to 2,600, N up to
9,000, K up to 8,320, groups of up to four matrices; MoE with up to 64
experts, top-k up to 8, ragged hidden and inter sizes), so the cases land on
every launch plan with ragged edges."""

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs
from tests.helpers import GEMV_TOL, MFMA_TOL, rel_err

pytestmark = pytest.mark.gpu

FM = [(O.Q4, B.Q4_G32), (O.Q8, B.Q8_G32), (O.Q2, B.Q2_G32), (O.Q3, B.Q3_G32), (O.Q5, B.Q5_G32),
      (O.Q6, B.Q6_G32), (O.F16, B.F16), (O.BF16, B.BF16)]


def _dev(w, bf):
    return B.qm_repack(B.qm_quantise(torch.from_numpy(np.ascontiguousarray(w)).cuda(), bf), B.LAYOUT_DEVICE)


def _logu(rng, lo, hi):
    return int(np.exp(rng.uniform(np.log(lo), np.log(hi))))


def _ref_cols(w, cols, x_rows, of):
    q, s = O.quantise(w[cols], of)
    return O.gemm(O.pack(q, of), s, of, x_rows)


@pytest.mark.parametrize("case", range(48))
def test_random_gemv_gemm(case):
    rng = np.random.default_rng(1000 + case)
    of, bf = FM[case % len(FM)]
    m = 1 if case % 3 == 0 else _logu(rng, 2, 2600)
    n, k = _logu(rng, 1, 9000), 32 * _logu(rng, 1, 260)
    w = inputs.weights_np(int(rng.integers(1 << 30)), (n, k))
    x = inputs.activations_np(int(rng.integers(1 << 30)), (m, k))
    y = B.qmatmul_gemm(_dev(w, bf), torch.from_numpy(x).cuda()).cpu().numpy()
    rows = np.unique(rng.choice(m, min(m, 12), replace=False))
    cols = np.unique(np.concatenate([rng.choice(n, min(n, 48), replace=False), [n - 1]]))
    err = rel_err(y[np.ix_(rows, cols)], _ref_cols(w, cols, x[rows], of))
    assert err <= (GEMV_TOL if m == 1 else MFMA_TOL), (m, n, k, err)


@pytest.mark.parametrize("case", range(16))
def test_random_gemm_grouped(case):
    rng = np.random.default_rng(2000 + case)
    of, bf = FM[case % len(FM)]
    m, k = _logu(rng, 1, 2600), 32 * _logu(rng, 1, 200)
    ns = [_logu(rng, 1, 6000) for _ in range(int(rng.integers(1, 5)))]
    ws = [inputs.weights_np(int(rng.integers(1 << 30)), (n, k)) for n in ns]
    x = inputs.activations_np(int(rng.integers(1 << 30)), (m, k))
    ys = B.qmatmul_gemm_grouped([_dev(w, bf) for w in ws], torch.from_numpy(x).cuda())
    rows = np.unique(rng.choice(m, min(m, 8), replace=False))
    for w, n, yv in zip(ws, ns, ys):
        cols = np.unique(np.concatenate([rng.choice(n, min(n, 24), replace=False), [n - 1]]))
        err = rel_err(yv.cpu().numpy()[np.ix_(rows, cols)], _ref_cols(w, cols, x[rows], of))
        assert err <= (GEMV_TOL if m == 1 else MFMA_TOL), (m, ns, k, err)


@pytest.mark.parametrize("case", range(12))
def test_random_moe(case):
    rng = np.random.default_rng(3000 + case)
    E = _logu(rng, 2, 64)
    top_k = int(rng.integers(1, min(8, E) + 1))
    m, H, I = _logu(rng, 1, 700), 32 * _logu(rng, 1, 24), 32 * _logu(rng, 1, 16)
    gw = inputs.weights_np(int(rng.integers(1 << 30)), (E, I, H))
    uw = inputs.weights_np(int(rng.integers(1 << 30)), (E, I, H))
    dw = inputs.weights_np(int(rng.integers(1 << 30)), (E, H, I))
    x = inputs.activations_np(int(rng.integers(1 << 30)), (m, H))
    lg = inputs.logits_np(int(rng.integers(1 << 30)), (m, E))
    r = B.qmoe_route(torch.from_numpy(lg).cuda(), top_k)
    y = B.qmoe_grouped_gemm(_dev(gw, B.Q4_G32), _dev(uw, B.Q4_G32), _dev(dw, B.Q4_G32),
                            torch.from_numpy(x).cuda(), r).cpu().numpy()
    packed = []
    for a in (gw, uw, dw):
        q, s = O.quantise(a.reshape(-1, a.shape[-1]), O.Q4)
        packed += [O.pack(q, O.Q4).reshape(E, a.shape[1], -1), s.reshape(E, a.shape[1], -1)]
    ref = O.moe_layer(x, lg, top_k, *packed)[0]
    assert rel_err(y, ref) <= MFMA_TOL, (E, top_k, m, H, I)
