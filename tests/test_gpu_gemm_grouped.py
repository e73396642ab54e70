"""GPU parity of the grouped prefill GEMM (qmatmul_gemm_grouped) with the
oracle, and with one qmatmul_gemm call per matrix."""

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs, workloads
from tests.helpers import MFMA_TOL, rel_err

pytestmark = pytest.mark.gpu


def _case(m, k, ns, seed, sample=None):
    ws_np = [inputs.weights_np(inputs.seed_for(3, seed, "q", i), (n, k)) for i, n in enumerate(ns)]
    x = inputs.activations_np(inputs.seed_for(3, seed, "x"), (m, k))
    wd = [B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), B.Q4_G32), B.LAYOUT_DEVICE) for w in ws_np]
    xt = torch.from_numpy(x).cuda()
    ys = B.qmatmul_gemm_grouped(wd, xt)
    rng = np.random.default_rng(seed)
    for i, (w, n) in enumerate(zip(ws_np, ns)):
        y = ys[i].cpu().numpy()
        rows = np.arange(m) if sample is None else np.unique(np.concatenate([rng.choice(m, sample, replace=False), [0, m - 1]]))
        cols = np.arange(n) if sample is None else np.unique(np.concatenate([rng.choice(n, min(n, 8 * sample), replace=False), [0, n - 1]]))
        q, s = O.quantise(w[cols], O.Q4)
        ref = O.gemm(O.pack(q, O.Q4), s, O.Q4, x[rows])
        assert rel_err(y[np.ix_(rows, cols)], ref) <= MFMA_TOL, i
        single = B.qmatmul_gemm(wd[i], xt).cpu().numpy()
        assert rel_err(y, single.astype(np.float64)) <= 1e-5, i


def test_grouped_qkv_llama_1b_layer_m128():
    """Llama-3.2-1B q/k/v (2048 -> 2048, 512, 512) sharing X, M = 128."""
    _case(128, 2048, [2048, 512, 512], 1, sample=10)


def test_grouped_gate_up_m512():
    _case(512, 2048, [8192, 8192], 2, sample=10)


def test_grouped_ragged_four_matrices():
    """Four matrices with ragged row counts, ragged M and K = 32 * odd."""
    _case(70, 160, [1, 65, 200, 130], 3)


def test_grouped_m1_runs_the_grouped_gemv():
    _case(1, 1024, [2048, 1024, 1024], 4)


def test_grouped_large_m_uses_big_tiles():
    """M = 2048: the 128 x 256 tile across a matrix boundary."""
    _case(2048, 256, [4160, 4096], 5, sample=12)
