"""GPU parity of the grouped decode GEMV (qmatmul_gemv_grouped) with the
oracle, and with one qmatmul_gemv call per matrix."""

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs
from tests.helpers import GEMV_TOL, rel_err

pytestmark = pytest.mark.gpu

FMTS = [(O.Q4, B.Q4_G32), (O.Q8, B.Q8_G32)]


def _case(ofmt, bfmt, k, ns, shared_x, seed):
    ws_np = [inputs.weights_np(inputs.seed_for(7, seed, "q", i), (n, k)) for i, n in enumerate(ns)]
    if shared_x:
        x = inputs.activations_np(inputs.seed_for(7, seed, "x"), (k,))
        xs_np = [x] * len(ns)
    else:
        xs_np = [inputs.activations_np(inputs.seed_for(7, seed, "x", i), (k,)) for i in range(len(ns))]
    wd = [B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), bfmt), B.LAYOUT_DEVICE) for w in ws_np]
    xt = {}
    xs = [xt.setdefault(id(x), torch.from_numpy(x).cuda()) for x in xs_np]
    ys = B.qmatmul_gemv_grouped(wd, xs)
    for i, (w, x) in enumerate(zip(ws_np, xs_np)):
        q, s = O.quantise(w, ofmt)
        ref = O.gemv(O.pack(q, ofmt), s, ofmt, x)
        y = ys[i].cpu().numpy()
        assert rel_err(y, ref) <= GEMV_TOL, i
        single = B.qmatmul_gemv(wd[i], xs[i]).cpu().numpy()
        assert rel_err(y, single.astype(np.float64)) <= 1e-5, i


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
def test_grouped_qkv_shared_x(ofmt, bfmt):
    """Qwen3-0.6B q/k/v projections (1024 -> 2048, 1024, 1024) sharing x."""
    _case(ofmt, bfmt, 1024, [2048, 1024, 1024], True, 1)


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
def test_grouped_gate_up_shared_x(ofmt, bfmt):
    """Qwen3-0.6B gate and up projections (1024 -> 3072 each) sharing x."""
    _case(ofmt, bfmt, 1024, [3072, 3072], True, 2)


@pytest.mark.parametrize("ofmt,bfmt", FMTS)
def test_grouped_ragged_eight_distinct_x(ofmt, bfmt):
    """Eight matrices with ragged row counts (1 .. 700) and distinct inputs."""
    _case(ofmt, bfmt, 96, [1, 63, 64, 65, 130, 700, 5, 200], False, 3)


def test_grouped_single_entry_and_large_k():
    _case(O.Q4, B.Q4_G32, 8192, [100], False, 4)
    _case(O.Q4, B.Q4_G32, 5120, [300, 70], True, 5)


def test_grouped_many_rows_uses_per_matrix_launches():
    """Total rows >= 64 per CU: the panel kernel, one launch per matrix."""
    _case(O.Q4, B.Q4_G32, 256, [9000, 8000], False, 6)


def test_grouped_empty_entry_is_noop():
    wd = [B.empty_qweight(B.Q4_G32, B.LAYOUT_DEVICE, 1, 0, 64),
          B.qm_repack(B.qm_quantise(torch.ones(70, 64, device="cuda"), B.Q4_G32), B.LAYOUT_DEVICE)]
    x = torch.ones(64, dtype=torch.float16, device="cuda")
    y0 = torch.full((4,), 7.0, device="cuda")
    y1 = torch.zeros(70, device="cuda")
    B.qmatmul_gemv_grouped(wd, [x, x], outs=[y0, y1])
    assert torch.all(y0 == 7.0)
    assert torch.equal(y1, B.qmatmul_gemv(wd[1], x))
