"""The allocation-free MoE entry point (qmoe_grouped_gemm_noalloc) against
the workspace one (qmoe_grouped_gemm) on the same inputs: three calls in a
row on the library's shared scratch, the first at the largest size it
accepts, each later one smaller, every output bit for bit equal to the
workspace call's (same kernels, same launch plan)."""

import numpy as np
import pytest
import torch

from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs

pytestmark = pytest.mark.gpu


def _experts(seed, e, hidden, inter):
    mk = lambda t, sh: B.qm_repack(B.qm_quantise(inputs.weights_dev(inputs.seed_for(seed, 0, t), sh), B.Q4_G32),
                                   B.LAYOUT_DEVICE)
    return mk("gate", (e, inter, hidden)), mk("up", (e, inter, hidden)), mk("down", (e, hidden, inter))


def test_noalloc_matches_workspace_entry_point():
    e, k, hidden, inter = 16, 8, 2048, 768
    wg, wu, wd = _experts(61, e, hidden, inter)
    for m in (744, 300, 37):              # 744: the largest m whose scratch fits
        print(f"noalloc m={m}", flush=True)
        assert B.qmoe_workspace_bytes(m, e, k, hidden, inter) <= B.NOALLOC_SCRATCH_BYTES
        x = inputs.activations_dev(inputs.seed_for(61, m, "x"), (m, hidden))
        logits = inputs.logits_dev(inputs.seed_for(61, m, "logits"), (m, e))
        r = B.qmoe_route(logits, k)
        y_ws = B.qmoe_grouped_gemm(wg, wu, wd, x, r)
        y_na = B.qmoe_grouped_gemm_noalloc(wg, wu, wd, x, r)
        torch.cuda.synchronize()
        assert torch.isfinite(y_na).all()
        assert torch.equal(y_na, y_ws), m
    with pytest.raises(B.QmError) as err:
        m = 745
        x = inputs.activations_dev(1, (m, hidden))
        B.qmoe_grouped_gemm_noalloc(wg, wu, wd, x, B.qmoe_route(inputs.logits_dev(2, (m, e)), k))
    assert err.value.status == 6
