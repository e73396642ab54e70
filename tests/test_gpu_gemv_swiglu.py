"""GPU parity of the SwiGLU gate/up GEMV pair (qmatmul_gemv_swiglu) with the
oracle: h = silu(Wg' x) * (Wu' x) in one launch."""

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs
from tests.helpers import GEMV_TOL, rel_err

pytestmark = pytest.mark.gpu

FMTS = [(O.Q4, B.Q4_G32), (O.Q8, B.Q8_G32)]


def _pair(n, k, ofmt, bfmt, tag):
    wg = inputs.weights_np(inputs.seed_for(tag, n, "gate"), (n, k))
    wu = inputs.weights_np(inputs.seed_for(tag, n, "up"), (n, k))
    x = inputs.activations_np(inputs.seed_for(tag, n, "x"), (k,))
    dev = [B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), bfmt), B.LAYOUT_DEVICE) for w in (wg, wu)]
    (gq, gs), (uq, us) = O.quantise(wg, ofmt), O.quantise(wu, ofmt)
    ref = O.gemv_swiglu(O.pack(gq, ofmt), gs, O.pack(uq, ofmt), us, ofmt, x)
    return dev, x, ref


# Ragged N, 4/8/16/32-row workgroups, x in LDS (K <= 4096) and read from
# global memory (K > 4096), and matrices big enough for the panel plan
# (N >= 16384), which the pair runs with 32-row workgroups.
@pytest.mark.parametrize("ofmt,bfmt", FMTS)
@pytest.mark.parametrize("n,k", [(1, 32), (65, 96), (200, 1024), (1000, 2048), (130, 3072),
                                 (64, 8192), (70, 20000), (3072, 1024), (4100, 1024), (16448, 256)])
def test_gemv_swiglu_parity(ofmt, bfmt, n, k):
    (wg, wu), x, ref = _pair(n, k, ofmt, bfmt, 2)
    h = B.qmatmul_gemv_swiglu(wg, wu, torch.from_numpy(x).cuda()).cpu().numpy()
    assert rel_err(h, ref) <= GEMV_TOL
    assert rel_err(h, ref) <= 1e-5


@pytest.mark.parametrize("n,k", [(3072, 1024), (8192, 3072)])
def test_gemv_swiglu_ffn_shapes_match_two_gemvs(n, k):
    """Feed-forward shapes (Qwen3-0.6B and Llama-3.2-3B gate/up): the fused
    pair equals the oracle, and it agrees with two separate GEMVs whose
    outputs are combined on the host with the same SiLU."""
    (wg, wu), x, ref = _pair(n, k, O.Q4, B.Q4_G32, 3)
    xt = torch.from_numpy(x).cuda()
    h = B.qmatmul_gemv_swiglu(wg, wu, xt)
    assert rel_err(h.cpu().numpy(), ref) <= GEMV_TOL
    a = B.qmatmul_gemv(wg, xt).double()
    b = B.qmatmul_gemv(wu, xt).double()
    two = (a / (1 + torch.exp(-a)) * b).cpu().numpy()
    assert rel_err(h.cpu().numpy(), two) <= 1e-5
    assert torch.equal(h, B.qmatmul_gemv_swiglu(wg, wu, xt))        # deterministic


def test_gemv_swiglu_extreme_gate_values():
    """Large positive and negative gate sums: silu saturates to the gate
    value and to zero without producing NaN or inf."""
    n, k = 96, 64
    rng = np.random.default_rng(5)
    wg = np.zeros((n, k), np.float32)
    wg[:, 0] = np.linspace(-120.0, 120.0, n)
    wu = rng.standard_normal((n, k)).astype(np.float32)
    x = np.zeros(k, np.float16)
    x[0], x[1] = 1.0, 0.5
    dev = [B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), B.Q8_G32), B.LAYOUT_DEVICE) for w in (wg, wu)]
    h = B.qmatmul_gemv_swiglu(dev[0], dev[1], torch.from_numpy(x).cuda()).cpu().numpy()
    (gq, gs), (uq, us) = O.quantise(wg, O.Q8), O.quantise(wu, O.Q8)
    ref = O.gemv_swiglu(O.pack(gq, O.Q8), gs, O.pack(uq, O.Q8), us, O.Q8, x)
    assert np.all(np.isfinite(h))
    assert rel_err(h, ref) <= 1e-5
