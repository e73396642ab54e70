"""GPU parity of the MFMA GEMM with Q8 weights (qmatmul_gemm and
qmatmul_gemm_grouped on QM_Q8_G32) with the oracle."""

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs, workloads
from tests.helpers import GEMV_TOL, MFMA_TOL, rel_err

pytestmark = pytest.mark.gpu


def _device_weight(w_np):
    w = torch.from_numpy(np.ascontiguousarray(w_np)).cuda()
    return B.qm_repack(B.qm_quantise(w, B.Q8_G32), B.LAYOUT_DEVICE)


def _ref(w, x):
    q, s = O.quantise(w, O.Q8)
    return O.gemm(O.pack(q, O.Q8), s, O.Q8, x)


# Every Q8 tile: 64 x 256 (two shapes), 64 x 128 split-K, one-panel split-K
# slices of 64 and 32 rows; ragged M, N and K (K = 32 * odd, 8224, 4128).
@pytest.mark.parametrize("m,n,k", [(2, 64, 32), (5, 65, 96), (127, 130, 160), (129, 64, 64),
                                   (64, 256, 1024), (300, 200, 2048), (513, 384, 256),
                                   (128, 512, 2048), (33, 1000, 8192), (2048, 2048, 96),
                                   (70, 640, 8224), (200, 4096, 4128)])
def test_gemm_q8_parity(m, n, k):
    w = inputs.weights_np(inputs.seed_for(5, n, "gate"), (n, k))
    x = inputs.activations_np(inputs.seed_for(5, m, "x"), (m, k))
    y = B.qmatmul_gemm(_device_weight(w), torch.from_numpy(x).cuda()).cpu().numpy()
    err = rel_err(y, _ref(w, x))
    assert err <= MFMA_TOL
    assert err <= 2e-3, err                  # fp16 weight rounding only


def test_gemm_q8_large_ragged_sampled():
    """2000 x 4100 x 96: the shape class where Q4 takes 128 x 256 tiles and
    Q8 64 x 256; sampled rows and columns across tile boundaries."""
    m, n, k = 2000, 4100, 96
    w = inputs.weights_np(inputs.seed_for(5, n, "up", 3), (n, k))
    x = inputs.activations_np(inputs.seed_for(5, m, "x", 3), (m, k))
    y = B.qmatmul_gemm(_device_weight(w), torch.from_numpy(x).cuda()).cpu().numpy()
    rng = np.random.default_rng(83)
    rows = np.unique(np.concatenate([rng.choice(m, 40, replace=False), [0, 63, 64, 1983, 1984, m - 1]]))
    cols = np.unique(np.concatenate([rng.choice(n, 300, replace=False), [0, 255, 256, 4095, 4096, n - 1]]))
    assert rel_err(y[np.ix_(rows, cols)], _ref(w[cols], x[rows])) <= MFMA_TOL


def test_gemm_q8_integer_grid_exact():
    """Integer weights in [-127, 127] with scale 1 (every group holds +-127)
    are exact in fp16; products and sums of small integers are exact in the
    fp32 accumulator.  Covers every byte value's unpacking."""
    rng = np.random.default_rng(18)
    m, n, k = 70, 190, 512
    w = rng.integers(-127, 128, size=(n, k))
    w[:, ::32] = 127
    w[:, 1::32] = -127
    x = rng.integers(-4, 5, size=(m, k)).astype(np.float16)
    y = B.qmatmul_gemm(_device_weight(w.astype(np.float32)), torch.from_numpy(x).cuda()).cpu().numpy()
    assert np.array_equal(y.astype(np.float64), _ref(w.astype(np.float32), x))


def test_gemm_q8_uses_fp16_rounded_weights():
    """X = identity rows: Y[i][n] is the fp16 operand fp16_RNE(s*q) of
    weight (n, i)."""
    n, k = 128, 64
    w = inputs.weights_np(15, (n, k))
    x = np.eye(k, dtype=np.float16)
    y = B.qmatmul_gemm(_device_weight(w), torch.from_numpy(x).cuda()).cpu().numpy()
    q, s = O.quantise(w, O.Q8)
    tile = O.dequantise_f16_tile_value(O.pack(q, O.Q8), s, O.Q8)
    assert np.array_equal(y.T.astype(np.float16).view(np.uint16), tile)


def test_gemm_q8_m1_matches_gemv_and_is_deterministic():
    n, k = 333, 1024
    w = inputs.weights_np(19, (n, k))
    x = inputs.activations_np(20, (1, k))
    wd = _device_weight(w)
    xt = torch.from_numpy(x).cuda()
    assert torch.equal(B.qmatmul_gemm(wd, xt)[0], B.qmatmul_gemv(wd, xt[0]))
    x2 = torch.from_numpy(inputs.activations_np(22, (257, k))).cuda()
    a = B.qmatmul_gemm(wd, x2)
    assert torch.equal(a, B.qmatmul_gemm(wd, x2))
    assert rel_err(a.cpu().numpy(), _ref(w, x2.cpu().numpy())) <= MFMA_TOL
    q, s = O.quantise(w, O.Q8)
    assert rel_err(B.qmatmul_gemv(wd, xt[0]).cpu().numpy(), O.gemv(O.pack(q, O.Q8), s, O.Q8, x[0])) <= GEMV_TOL


@pytest.mark.parametrize("m", [512, 2048])
def test_prefill_layer_q8_full_size_sampled(m):
    """Every projection of one Llama-3.2-1B layer in Q8 at full size;
    sampled output rows and columns."""
    rng = np.random.default_rng(m + 8)
    for li, (name, k, n) in enumerate(workloads.LLAMA32_1B_LAYER):
        w = inputs.weights_np(inputs.seed_for(3, 1, name), (n, k))
        x = inputs.activations_np(inputs.seed_for(3, 1, "x", li), (m, k))
        y = B.qmatmul_gemm(_device_weight(w), torch.from_numpy(x).cuda()).cpu().numpy()
        rows = np.unique(np.concatenate([rng.choice(m, 12, replace=False), [0, m - 1]]))
        cols = np.unique(np.concatenate([rng.choice(n, 150, replace=False), [0, n - 1]]))
        assert rel_err(y[np.ix_(rows, cols)], _ref(w[cols], x[rows])) <= MFMA_TOL, name


@pytest.mark.parametrize("m,k,ns", [(128, 2048, [2048, 512, 512]), (512, 2048, [8192, 8192]),
                                    (70, 160, [1, 65, 200, 130])])
def test_gemm_q8_grouped(m, k, ns):
    """Grouped Q8 GEMM: each entry against the oracle (sampled) and against
    its own qmatmul_gemm call."""
    ws = [inputs.weights_np(inputs.seed_for(5, m, "q", i), (n, k)) for i, n in enumerate(ns)]
    x = inputs.activations_np(inputs.seed_for(5, m, "x", 9), (m, k))
    wd = [_device_weight(w) for w in ws]
    xt = torch.from_numpy(x).cuda()
    ys = B.qmatmul_gemm_grouped(wd, xt)
    rng = np.random.default_rng(m)
    for i, (w, n) in enumerate(zip(ws, ns)):
        y = ys[i].cpu().numpy()
        rows = np.unique(np.concatenate([rng.choice(m, min(m, 10), replace=False), [0, m - 1]]))
        cols = np.unique(np.concatenate([rng.choice(n, min(n, 80), replace=False), [0, n - 1]]))
        assert rel_err(y[np.ix_(rows, cols)], _ref(w[cols], x[rows])) <= MFMA_TOL, i
        single = B.qmatmul_gemm(wd[i], xt).cpu().numpy()
        assert rel_err(y, single.astype(np.float64)) <= 1e-5, i
