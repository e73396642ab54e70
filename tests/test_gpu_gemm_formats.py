"""GPU parity of the MFMA GEMM with Q2/Q3/Q5/Q6 and F16/BF16 weights
(qmatmul_gemm and qmatmul_gemm_grouped) with the oracle (Sec. 3.3: one GEMM
per format for M > 1; Sec. 4.1: the eight formats)."""

import ctypes

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs
from tests.helpers import MFMA_TOL, rel_err

pytestmark = pytest.mark.gpu

FMTS = [(O.Q2, B.Q2_G32), (O.Q3, B.Q3_G32), (O.Q5, B.Q5_G32), (O.Q6, B.Q6_G32),
        (O.F16, B.F16), (O.BF16, B.BF16)]


def _device_weight(w_np, bfmt):
    w = torch.from_numpy(np.ascontiguousarray(w_np)).cuda()
    return B.qm_repack(B.qm_quantise(w, bfmt), B.LAYOUT_DEVICE)


def _ref(w, x, ofmt):
    q, s = O.quantise(w, ofmt)
    return O.gemm(O.pack(q, ofmt), s, ofmt, x)


# Every tile of the plan: 128 x 256 (2048 x 4096), 64 x 256, 64 x 128
# split-K (500 x 3000 x 2080), one-panel split-K with 64 and 32 rows;
# ragged M, N, K.
@pytest.mark.parametrize("ofmt,bfmt", FMTS)
@pytest.mark.parametrize("m,n,k", [(2, 64, 32), (5, 65, 96), (127, 130, 160), (300, 200, 2048),
                                   (33, 1000, 8192), (2048, 2048, 96), (200, 4096, 4128),
                                   (500, 3000, 2080), (2000, 4100, 64)])
def test_gemm_formats_parity(ofmt, bfmt, m, n, k):
    w = inputs.weights_np(inputs.seed_for(6, n, "gate", ofmt), (n, k))
    x = inputs.activations_np(inputs.seed_for(6, m, "x", ofmt), (m, k))
    y = B.qmatmul_gemm(_device_weight(w, bfmt), torch.from_numpy(x).cuda()).cpu().numpy()
    if m * n > 600_000:
        rng = np.random.default_rng(m + n)
        rows = np.unique(np.concatenate([rng.choice(m, 40, replace=False), [0, 63, 64, 127, 128, m - 1]]))
        cols = np.unique(np.concatenate([rng.choice(n, 300, replace=False), [0, 255, 256, n - 1]]))
        err = rel_err(y[np.ix_(rows, cols)], _ref(w[cols], x[rows], ofmt))
    else:
        err = rel_err(y, _ref(w, x, ofmt))
    assert err <= MFMA_TOL
    assert err <= 2e-3, err


# Every output checked (no sampling) on tiles whose K slices end with steps
# after the main loop, where the loads of a workgroup's last steps must all
# have landed before their LDS tiles are read: 64 x 64 with 4-way split-K
# (512 x 2048 x 2048), 64 x 128 with 2-way split-K, 128 x 256, and 64 x 64
# with 8-way split-K over a ragged K.
@pytest.mark.parametrize("ofmt,bfmt", [(O.Q4, B.Q4_G32), (O.Q8, B.Q8_G32), (O.F16, B.F16), (O.BF16, B.BF16)])
@pytest.mark.parametrize("m,n,k", [(512, 2048, 2048), (500, 3000, 2080), (2000, 4100, 64), (200, 4096, 4128)])
def test_gemm_every_output_last_k_steps(ofmt, bfmt, m, n, k):
    w = inputs.weights_np(inputs.seed_for(7, n, "up", ofmt), (n, k))
    x = inputs.activations_np(inputs.seed_for(7, m, "x", ofmt), (m, k))
    y = B.qmatmul_gemm(_device_weight(w, bfmt), torch.from_numpy(x).cuda()).cpu().numpy()
    err = rel_err(y, _ref(w, x, ofmt))
    assert err <= 2e-3, err


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
@pytest.mark.parametrize("m,n,k", [(70, 190, 512), (1100, 2048, 64)])
def test_gemm_formats_integer_grid_exact(ofmt, bfmt, m, n, k):
    """Scale-1 integer weights over every code in [-qmax, qmax] (F16/BF16:
    integers in [-64, 64], exact in both) and small integer X: the fp32
    result is exact (B through registers and LDS)."""
    rng = np.random.default_rng(40 + ofmt)
    qm = O.QMAX.get(ofmt, 64)
    w = rng.integers(-qm, qm + 1, size=(n, k))
    w[:, ::32] = qm
    x = rng.integers(-4, 5, size=(m, k)).astype(np.float16)
    y = B.qmatmul_gemm(_device_weight(w.astype(np.float32), bfmt), torch.from_numpy(x).cuda()).cpu().numpy()
    assert np.array_equal(y.astype(np.float64), _ref(w.astype(np.float32), x, ofmt))


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
def test_gemm_formats_use_fp16_rounded_weights(ofmt, bfmt):
    n, k = 128, 64
    w = inputs.weights_np(25 + ofmt, (n, k))
    x = np.eye(k, dtype=np.float16)
    y = B.qmatmul_gemm(_device_weight(w, bfmt), torch.from_numpy(x).cuda()).cpu().numpy()
    q, s = O.quantise(w, ofmt)
    assert np.array_equal(y.T.astype(np.float16).view(np.uint16), O.dequantise_f16_tile_value(O.pack(q, ofmt), s, ofmt))


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
def test_gemm_formats_grouped(ofmt, bfmt):
    m, k, ns = 512, 2048, [2048, 512, 512]
    ws = [inputs.weights_np(inputs.seed_for(6, 1, "q", i + 10 * ofmt), (n, k)) for i, n in enumerate(ns)]
    x = inputs.activations_np(inputs.seed_for(6, 2, "x", ofmt), (m, k))
    wd = [_device_weight(w, bfmt) for w in ws]
    xt = torch.from_numpy(x).cuda()
    ys = B.qmatmul_gemm_grouped(wd, xt)
    rng = np.random.default_rng(ofmt)
    for i, (w, n) in enumerate(zip(ws, ns)):
        y = ys[i].cpu().numpy()
        rows = np.unique(np.concatenate([rng.choice(m, 10, replace=False), [0, m - 1]]))
        cols = np.unique(np.concatenate([rng.choice(n, 80, replace=False), [0, n - 1]]))
        assert rel_err(y[np.ix_(rows, cols)], _ref(w[cols], x[rows], ofmt)) <= MFMA_TOL, i
        assert rel_err(y, B.qmatmul_gemm(wd[i], xt).cpu().numpy().astype(np.float64)) <= 1e-5, i


@pytest.mark.parametrize("bfmt", [B.F16, B.BF16])
def test_gemm_float_formats_m1_runs_the_gemv(bfmt):
    w = _device_weight(inputs.weights_np(3, (64, 64)), bfmt)
    x = torch.from_numpy(inputs.activations_np(4, (2, 64))).cuda()
    y = torch.empty((2, 64), device="cuda")
    st = B.lib().qmatmul_gemm(ctypes.byref(w.c()), ctypes.c_void_p(x.data_ptr()), 2, ctypes.c_void_p(y.data_ptr()), None)
    assert st == 0, B.qm_last_error()
    y1 = B.qmatmul_gemm(w, x[:1])                                        # m = 1 runs the GEMV
    assert torch.equal(y1[0], B.qmatmul_gemv(w, x[0]))


def test_gemm_bf16_weights_reach_the_mfma_as_fp16():
    """BF16 weights over 2^-26 .. 2^15 times the identity: every output is
    the weight's value rounded to nearest-even fp16, exact where it lies in
    fp16's normal range, a subnormal (or zero) below it."""
    n, k = 192, 96
    rng = np.random.default_rng(77)
    w = (np.sign(rng.standard_normal((n, k))) * np.exp2(rng.uniform(-26, 15, (n, k)))).astype(np.float32)
    x = np.eye(k, dtype=np.float16)
    y = B.qmatmul_gemm(_device_weight(w, B.BF16), torch.from_numpy(x).cuda()).cpu().numpy()
    bits, _ = O.quantise(w, O.BF16)
    want = O.fp16_value(O.dequantise_f16_tile_value(O.pack(bits, O.BF16), None, O.BF16))
    # Compared as values: a weight that rounds to -0 gives +0 once the
    # other k's zero products are added.
    assert np.array_equal(y.T.astype(np.float64), want.astype(np.float64))
    small = np.abs(O.bf16_value(bits)) < 2.0 ** -14
    assert small.any() and (~small).any()
    assert np.array_equal(y.T[~small].astype(np.float64), O.bf16_value(bits)[~small].astype(np.float64))


# F16 / BF16 weights at the Llama-3.2-1B prefill shapes (gate 2048 -> 8192 and
# down 8192 -> 2048) at M = 512 and 2048: sampled rows and columns against the
# oracle, every tile kind these sizes get from the plan.
@pytest.mark.parametrize("ofmt,bfmt", [(O.F16, B.F16), (O.BF16, B.BF16)])
@pytest.mark.parametrize("m,n,k", [(512, 8192, 2048), (2048, 2048, 8192), (512, 2048, 8192)])
def test_gemm_float_formats_full_size_sampled(ofmt, bfmt, m, n, k):
    w = inputs.weights_np(inputs.seed_for(3, 0, "gate" if n == 8192 else "down", ofmt), (n, k))
    x = inputs.activations_np(inputs.seed_for(3, m, "x", ofmt), (m, k))
    y = B.qmatmul_gemm(_device_weight(w, bfmt), torch.from_numpy(x).cuda()).cpu().numpy()
    rng = np.random.default_rng(m + n + ofmt)
    rows = np.unique(np.concatenate([rng.choice(m, 24, replace=False), [0, 127, 128, m - 1]]))
    cols = np.unique(np.concatenate([rng.choice(n, 200, replace=False), [0, 63, 64, 255, 256, n - 1]]))
    err = rel_err(y[np.ix_(rows, cols)], _ref(w[cols], x[rows], ofmt))
    assert err <= 2e-3, err
