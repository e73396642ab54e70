"""GPU parity of the Q4 MFMA GEMM (qmatmul_gemm) with the oracle."""

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
    return B.qm_repack(B.qm_quantise(w, B.Q4_G32), B.LAYOUT_DEVICE)


@pytest.mark.parametrize("m,n,k", [(2, 64, 32), (5, 65, 96), (127, 130, 160), (129, 64, 64),
                                   (64, 256, 1024), (300, 200, 2048), (513, 384, 256),
                                   (128, 512, 2048), (33, 1000, 8192),
                                   (70, 640, 8224), (200, 4096, 4128)])   # 8-way split-K, ragged K slices
def test_gemm_parity(m, n, k):
    w = inputs.weights_np(inputs.seed_for(3, n, "gate"), (n, k))
    x = inputs.activations_np(inputs.seed_for(3, m, "x"), (m, k))
    wd = _device_weight(w)
    y = B.qmatmul_gemm(wd, torch.from_numpy(x).cuda()).cpu().numpy()
    q, s = O.quantise(w, O.Q4)
    ref = O.gemm(O.pack(q, O.Q4), s, O.Q4, x)
    err = rel_err(y, ref)
    assert err <= MFMA_TOL
    assert err <= 2e-3, err                  # fp16 weight rounding only: ~3e-4 expected


def test_gemm_large_ragged_sampled():
    """A large shape (the 128 x 256 tile at two workgroups per CU), ragged in
    every dimension: 2000 rows, 8000 columns, K = 96 (a half-empty last K
    step).  The oracle recomputes sampled rows and columns, including both
    sides of tile boundaries."""
    m, n, k = 2000, 8000, 96
    w = inputs.weights_np(inputs.seed_for(3, n, "gate", 256), (n, k))
    x = inputs.activations_np(inputs.seed_for(3, m, "x", 256), (m, k))
    wd = _device_weight(w)
    y = B.qmatmul_gemm(wd, torch.from_numpy(x).cuda()).cpu().numpy()
    rng = np.random.default_rng(256)
    rows = np.unique(np.concatenate([rng.choice(m, 40, replace=False), [0, 127, 128, 1919, 1920, m - 1]]))
    cols = np.unique(np.concatenate([rng.choice(n, 300, replace=False), [0, 255, 256, 7935, 7936, n - 1]]))
    q, s = O.quantise(w[cols], O.Q4)
    ref = O.gemm(O.pack(q, O.Q4), s, O.Q4, x[rows])
    assert rel_err(y[np.ix_(rows, cols)], ref) <= MFMA_TOL


def test_gemm_two_panel_split_k_ragged_sampled():
    """A shape the 64 x 128 two-way split-K tile takes: 500 rows, 3000
    columns (a half-filled last panel pair), K = 2080 (33 K steps: the second
    slice has one step past the end).  Sampled rows and columns."""
    m, n, k = 500, 3000, 2080
    w = inputs.weights_np(inputs.seed_for(3, n, "up", 2), (n, k))
    x = inputs.activations_np(inputs.seed_for(3, m, "x", 2), (m, k))
    wd = _device_weight(w)
    y = B.qmatmul_gemm(wd, torch.from_numpy(x).cuda()).cpu().numpy()
    rng = np.random.default_rng(22)
    rows = np.unique(np.concatenate([rng.choice(m, 30, replace=False), [0, 63, 64, 447, 448, m - 1]]))
    cols = np.unique(np.concatenate([rng.choice(n, 200, replace=False), [0, 127, 128, 2943, 2944, n - 1]]))
    q, s = O.quantise(w[cols], O.Q4)
    ref = O.gemm(O.pack(q, O.Q4), s, O.Q4, x[rows])
    assert rel_err(y[np.ix_(rows, cols)], ref) <= MFMA_TOL


def test_gemm_integer_grid_exact():
    """Integer weights with scale 1 are exact in fp16, products and sums of
    small integers are exact in the fp32 MFMA accumulator."""
    rng = np.random.default_rng(8)
    m, n, k = 70, 190, 512
    w = rng.integers(-7, 8, size=(n, k))
    w[:, ::32] = -7
    x = rng.integers(-4, 5, size=(m, k)).astype(np.float16)
    wd = _device_weight(w.astype(np.float32))
    y = B.qmatmul_gemm(wd, torch.from_numpy(x).cuda()).cpu().numpy()
    q, s = O.quantise(w.astype(np.float32), O.Q4)
    assert np.array_equal(y.astype(np.float64), O.gemm(O.pack(q, O.Q4), s, O.Q4, x))


def test_gemm_uses_fp16_rounded_weights():
    """X = identity rows: Y[i][n] is the fp16 operand value fp16_RNE(s*q) of
    weight (n, i) -- the rounding the header documents."""
    n, k = 128, 64
    w = inputs.weights_np(5, (n, k))
    wd = _device_weight(w)
    x = np.eye(k, dtype=np.float16)
    y = B.qmatmul_gemm(wd, torch.from_numpy(x).cuda()).cpu().numpy()
    q, s = O.quantise(w, O.Q4)
    tile = O.dequantise_f16_tile_value(O.pack(q, O.Q4), s, O.Q4)
    assert np.array_equal(y.T.astype(np.float16).view(np.uint16), tile)


def test_gemm_m1_matches_gemv_and_is_deterministic():
    n, k = 333, 1024
    w = inputs.weights_np(9, (n, k))
    x = inputs.activations_np(10, (1, k))
    wd = _device_weight(w)
    xt = torch.from_numpy(x).cuda()
    y1 = B.qmatmul_gemm(wd, xt)
    y2 = B.qmatmul_gemv(wd, xt[0])
    assert torch.equal(y1[0], y2)
    x2 = torch.from_numpy(inputs.activations_np(12, (257, k))).cuda()
    a = B.qmatmul_gemm(wd, x2)
    b = B.qmatmul_gemm(wd, x2)
    assert torch.equal(a, b)
    q, s = O.quantise(w, O.Q4)
    assert rel_err(y1.cpu().numpy()[0], O.gemv(O.pack(q, O.Q4), s, O.Q4, x[0])) <= GEMV_TOL


@pytest.mark.parametrize("m", workloads.LLAMA32_1B_PREFILL["m_sweep"])
def test_prefill_layer_full_size_sampled(m):
    """Every projection of one Llama-3.2-1B layer at full size and M; the
    oracle recomputes sampled output rows and columns."""
    rng = np.random.default_rng(m)
    for li, (name, k, n) in enumerate(workloads.LLAMA32_1B_LAYER):
        w = inputs.weights_np(inputs.seed_for(3, 0, name), (n, k))
        x = inputs.activations_np(inputs.seed_for(3, 0, "x", li), (m, k))
        wd = _device_weight(w)
        y = B.qmatmul_gemm(wd, torch.from_numpy(x).cuda()).cpu().numpy()
        rows = np.unique(np.concatenate([rng.choice(m, 12, replace=False), [0, m - 1]]))
        cols = np.unique(np.concatenate([rng.choice(n, 150, replace=False), [0, n - 1]]))
        q, s = O.quantise(w[cols], O.Q4)
        ref = O.gemm(O.pack(q, O.Q4), s, O.Q4, x[rows])
        assert rel_err(y[np.ix_(rows, cols)], ref) <= MFMA_TOL, name
