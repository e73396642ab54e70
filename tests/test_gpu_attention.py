"""GPU parity of decode attention over a KV cache (qattn_decode) with the
oracle."""

import math

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from tests.helpers import rel_err

pytestmark = pytest.mark.gpu

ATTN_TOL = 2e-5    # fp32 scores, exp2 and sums against fp64


def _case(hq, hkv, d, length, max_len, seed, scale=None, poison=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((hq, d)).astype(np.float16)
    k = rng.standard_normal((hkv, max_len, d)).astype(np.float16)
    v = rng.standard_normal((hkv, max_len, d)).astype(np.float16)
    if poison and length < max_len:
        # rows past the length are not data: NaN there must not reach o
        k[:, length:] = np.float16(np.nan)
        v[:, length:] = np.float16(np.inf)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    o = B.qattn_decode(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda(),
                       length, scale).cpu().numpy()
    ref = O.attention_decode(q, k[:, :length], v[:, :length], length, np.float32(scale))
    return o, ref


# Group sizes 1-8, head_dim 64 and 128, a single row, ragged slices, lengths
# that need many slices, a full cache.
@pytest.mark.parametrize("hq,hkv,d,length,max_len", [
    (16, 8, 128, 1, 64), (16, 8, 128, 33, 64), (24, 8, 128, 1000, 1024), (32, 8, 64, 4097, 8192),
    (8, 8, 64, 100, 128), (64, 8, 128, 777, 1000), (12, 4, 128, 5000, 5000), (40, 8, 64, 31, 31),
    (14, 2, 128, 20000, 32768), (7, 1, 64, 3, 16)])
def test_attn_decode_parity(hq, hkv, d, length, max_len):
    o, ref = _case(hq, hkv, d, length, max_len, seed=hq * 1000 + length)
    assert np.all(np.isfinite(o))
    assert rel_err(o, ref) <= ATTN_TOL


def test_attn_decode_sharp_softmax():
    """Scale 1 on unit-variance q, k: scores spread over tens, so the slice
    maxima and the cross-slice merge decide the result."""
    o, ref = _case(16, 8, 128, 3000, 4096, seed=7, scale=1.0)
    assert rel_err(o, ref) <= ATTN_TOL


def test_attn_decode_long_context_sampled_heads():
    """Qwen3-0.6B attention shape (16 query heads, 8 KV heads, head_dim 128)
    at the longest supported context, 262144 rows (256 slices of 1024)."""
    hq, hkv, d, length = 16, 8, 128, 262144
    g = torch.Generator(device="cuda").manual_seed(11)
    q = torch.randn((hq, d), generator=g, device="cuda").half()
    k = torch.randn((hkv, length, d), generator=g, device="cuda").half()
    v = torch.randn((hkv, length, d), generator=g, device="cuda").half()
    o = B.qattn_decode(q, k, v, length, 1.0 / math.sqrt(d)).cpu().numpy()
    for kvh in (0, 5):
        ref = O.attention_decode(q[2 * kvh:2 * kvh + 2].cpu().numpy(), k[kvh:kvh + 1].cpu().numpy(),
                                 v[kvh:kvh + 1].cpu().numpy(), length, np.float32(1.0 / math.sqrt(d)))
        assert rel_err(o[2 * kvh:2 * kvh + 2], ref) <= ATTN_TOL


def test_attn_decode_deterministic_and_workspace_reuse():
    rng = np.random.default_rng(3)
    hq, hkv, d, n = 24, 8, 128, 2048
    q = torch.from_numpy(rng.standard_normal((hq, d)).astype(np.float16)).cuda()
    k = torch.from_numpy(rng.standard_normal((hkv, n, d)).astype(np.float16)).cuda()
    v = torch.from_numpy(rng.standard_normal((hkv, n, d)).astype(np.float16)).cuda()
    ws = torch.empty(B.qattn_decode_workspace_bytes(hq, d), dtype=torch.uint8, device="cuda")
    a = B.qattn_decode(q, k, v, n, 0.1, workspace=ws)
    b = B.qattn_decode(q, k, v, 17, 0.1, workspace=ws)          # another length in between
    c = B.qattn_decode(q, k, v, n, 0.1, workspace=ws)
    assert torch.equal(a, c)
    ref = O.attention_decode(q.cpu().numpy(), k.cpu().numpy()[:, :17], v.cpu().numpy()[:, :17], 17, np.float32(0.1))
    assert rel_err(b.cpu().numpy(), ref) <= ATTN_TOL
