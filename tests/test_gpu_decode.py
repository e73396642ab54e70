"""GPU parity of the decode-step glue kernels (embedding, RMSNorm with the
residual add, RoPE with the cache append, fp16 cast, greedy argmax) and of
whole decode steps of small dense decoders against the oracle's fp64
decode step."""

import math

import numpy as np
import pytest
import torch

from oracle import qmatmul_oracle as O
from paper_2607_00501_amd import binding as B
from paper_2607_00501_amd import inputs
from paper_2607_00501_amd.decoder import DecoderConfig, DenseDecoder, LayerWeights
from tests.helpers import GEMV_TOL, rel_err

pytestmark = pytest.mark.gpu


def _f16_bits(a):
    return np.asarray(a, dtype=np.float16).view(np.uint16)


# ---------------------------------------------------------------- glue kernels

# 16-byte-load tiles (hidden % 4 == 0, up to 8192), scalar register tiles
# (1026, 3002), and the two-pass loop (10000 is beyond the tiles, 12290 odd).
@pytest.mark.parametrize("rows,hidden", [(1, 1), (1, 96), (3, 1000), (1, 1024), (2, 4096), (1, 8192), (1, 1026),
                                         (2, 3002), (1, 10000), (1, 12290)])
@pytest.mark.parametrize("with_residual", [False, True])
def test_rmsnorm_parity(rows, hidden, with_residual):
    rng = np.random.default_rng(rows * 7 + hidden)
    x = (rng.standard_normal((rows, hidden)) * 3).astype(np.float32)
    r = rng.standard_normal((rows, hidden)).astype(np.float32)
    w = inputs.norm_weights_np(hidden, hidden)
    xd = torch.from_numpy(x).cuda()
    out = B.qdec_rmsnorm(xd, torch.from_numpy(w).cuda(), 1e-6,
                         residual=torch.from_numpy(r).cuda() if with_residual else None).cpu().numpy()
    xs = x.astype(np.float64) + (r if with_residual else 0.0)
    assert np.array_equal(xd.cpu().numpy(), (x + r) if with_residual else x)      # fp32 add written back
    for i in range(rows):
        ref = O.rmsnorm(xs[i], w, 1e-6)
        assert rel_err(out[i].astype(np.float64), ref) <= 1e-3                   # one fp16 rounding
        # at most one fp16 ulp away from the rounded oracle value
        diff = np.abs(_f16_bits(out[i]).astype(np.int32) - _f16_bits(O.f16(ref)).astype(np.int32))
        assert diff.max() <= 1


def test_rmsnorm_unaligned_row_uses_scalar_loads():
    """x starting 4 bytes into an allocation (not 16-byte aligned) gives the
    same result as an aligned copy."""
    rng = np.random.default_rng(3)
    big = torch.from_numpy(rng.standard_normal(2049).astype(np.float32)).cuda()
    res = torch.from_numpy(rng.standard_normal(2048).astype(np.float32)).cuda()
    w = torch.from_numpy(inputs.norm_weights_np(77, 2048)).cuda()
    x_un = big[1:]
    x_al = x_un.clone()
    a = B.qdec_rmsnorm(x_un, w, 1e-6, residual=res)
    b = B.qdec_rmsnorm(x_al, w, 1e-6, residual=res)
    assert torch.equal(x_un, x_al)
    assert (a.float() - b.float()).abs().max().item() <= 2.0 ** -10 * b.float().abs().max().item()


def test_rmsnorm_zero_rows_and_zero_vector():
    x = torch.zeros((1, 64), device="cuda")
    w = torch.ones(64, dtype=torch.float16, device="cuda")
    assert torch.all(B.qdec_rmsnorm(x, w, 1e-6) == 0)
    e = torch.empty((0, 64), device="cuda")
    assert B.qdec_rmsnorm(e, w, 1e-6).shape == (0, 64)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("pos,theta", [(0, 1e4), (7, 1e4), (1000, 5e5), (200_000, 1e6), (262_143, 1e6)])
def test_rope_append_parity(d, pos, theta):
    hq, hkv = 6, 2
    max_len = max(pos + 1, 16)
    rng = np.random.default_rng(pos + d)
    q = rng.standard_normal(hq * d).astype(np.float32)
    k = rng.standard_normal(hkv * d).astype(np.float32)
    v = rng.standard_normal(hkv * d).astype(np.float32)
    kc = torch.full((hkv, max_len, d), 0.5, dtype=torch.float16, device="cuda")
    vc = torch.full((hkv, max_len, d), -0.25, dtype=torch.float16, device="cuda")
    qo = B.qdec_rope_append(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda(),
                            pos, theta, kc, vc).cpu().numpy()
    ref_q = O.f16(O.rope(q.reshape(hq, d), pos, theta))
    ref_k = O.f16(O.rope(k.reshape(hkv, d), pos, theta))
    # fp32 rotation vs fp64, then one rounding each: one fp16 ulp (<= 2^-10
    # relative) plus the fp32 error of a near-cancelling a cos - b sin
    for got, want in ((qo, ref_q), (kc.cpu().numpy()[:, pos], ref_k)):
        got = got.astype(np.float64)
        assert np.all(np.abs(got - want) <= 2.0 ** -10 * np.abs(want) + 1e-6 * np.abs(want).max())
    kcn, vcn = kc.cpu().numpy(), vc.cpu().numpy()
    assert np.array_equal(vcn[:, pos], v.reshape(hkv, d).astype(np.float16))
    other = np.ones(max_len, bool)
    other[pos] = False
    assert np.all(kcn[:, other] == 0.5) and np.all(vcn[:, other] == -0.25)     # only row pos written


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("norms", [False, True])
def test_rope_append_table_gives_the_same_bits(d, norms):
    """qdec_rope_append reading qdec_rope_table's (cos, sin) writes the bits it
    writes computing each angle, with and without the per-head q/k norms."""
    hq, hkv, max_len, theta = 6, 2, 40_000, 1e6
    rng = np.random.default_rng(d + norms)
    q, k, v = (torch.from_numpy(rng.standard_normal(h * d).astype(np.float32)).cuda() for h in (hq, hkv, hkv))
    kw = {}
    if norms:
        kw = dict(q_norm=torch.from_numpy(rng.uniform(0.5, 1.5, d).astype(np.float16)).cuda(),
                  k_norm=torch.from_numpy(rng.uniform(0.5, 1.5, d).astype(np.float16)).cuda())
    tab = B.qdec_rope_table(max_len, d, theta)
    for pos in (0, 1, 77, 4095, 39_999):
        kc1 = torch.zeros((hkv, max_len, d), dtype=torch.float16, device="cuda")
        vc1, kc2, vc2 = torch.zeros_like(kc1), torch.zeros_like(kc1), torch.zeros_like(kc1)
        qa = B.qdec_rope_append(q, k, v, pos, theta, kc1, vc1, **kw)
        qb = B.qdec_rope_append(q, k, v, pos, theta, kc2, vc2, table=tab, **kw)
        assert torch.equal(qa, qb) and torch.equal(kc1, kc2) and torch.equal(vc1, vc2), pos


def test_cast_f16_bit_exact():
    rng = np.random.default_rng(9)
    x = np.concatenate([rng.standard_normal(1000).astype(np.float32) * 100,
                        np.array([65504.0, 65520.0, 65519.99, 1e6, -1e6, 6e-8, 3e-8, -2.9e-8, 1e-30, 0.0, -0.0,
                                  np.inf, -np.inf], np.float32),
                        # exact ties between neighbouring fp16 values round to even
                        (np.arange(1024, 1100, dtype=np.float32) + 0.5)])
    y = B.qdec_cast_f16(torch.from_numpy(x).cuda()).cpu().numpy()
    with np.errstate(over="ignore"):
        want = x.astype(np.float16)
    assert np.array_equal(_f16_bits(y), _f16_bits(want))
    assert B.qdec_cast_f16(torch.empty(0, device="cuda")).numel() == 0


@pytest.mark.parametrize("case", ["random", "ties", "nan", "allnan", "neginf", "one", "vocab"])
def test_argmax_parity(case):
    rng = np.random.default_rng(13)
    if case == "random":
        z = rng.standard_normal(5000).astype(np.float32)
    elif case == "ties":
        z = rng.standard_normal(300_000).astype(np.float32)
        z[[100_000, 5, 299_999, 1025]] = 50.0                # lowest index wins, across threads
    elif case == "nan":
        z = rng.standard_normal(4096).astype(np.float32)
        z[::3] = np.nan
    elif case == "allnan":
        z = np.full(777, np.nan, np.float32)
    elif case == "neginf":
        z = np.full(2000, -np.inf, np.float32)
        z[1999] = -1e30
    elif case == "one":
        z = np.array([-7.0], np.float32)
    else:
        z = rng.standard_normal(151_936).astype(np.float32)
    t = B.qdec_argmax(torch.from_numpy(z).cuda()).cpu().numpy()
    assert t.shape == (1,) and int(t[0]) == O.greedy_token(z)


def test_embed_gathers_rows_and_flags_bad_ids():
    table = inputs.activations_np(5, (1000, 256))
    td = torch.from_numpy(table).cuda()
    for t in (0, 999, 314):
        x = B.qdec_embed(td, torch.tensor([t], dtype=torch.int32, device="cuda")).cpu().numpy()
        assert np.array_equal(x, table[t].astype(np.float32))
    for t in (-1, 1000):
        x = B.qdec_embed(td, torch.tensor([t], dtype=torch.int32, device="cuda")).cpu().numpy()
        assert np.all(np.isnan(x))


# ---------------------------------------------------------------- decode steps

def _model(cfg: DecoderConfig, tag: int, fmts=(O.Q4, B.Q4_G32), interleave=False, qk_norm=False):
    """Seeded weights of a dense decoder, quantised on the device (library)
    and in the oracle from the same fp32 values."""
    ofmt, bfmt = fmts
    qd, kvd = cfg.n_q_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim

    def proj(name, li, n, k):
        w = inputs.weights_np(inputs.seed_for(tag, li, name), (n, k), sigma=1.0 / math.sqrt(k))
        wd = torch.from_numpy(w).cuda()
        if interleave and name in ("q", "k"):
            wd = B.rope_interleave_rows(wd, n // cfg.head_dim, cfg.head_dim)
        dev = B.qm_repack(B.qm_quantise(wd, bfmt), B.LAYOUT_DEVICE)
        q, s = O.quantise(w, ofmt)
        return dev, O.dequantise(O.pack(q, ofmt), s, ofmt).astype(np.float64)

    dev_layers, ref_layers = [], []
    for li in range(cfg.layers):
        shapes = dict(q=(qd, cfg.hidden), k=(kvd, cfg.hidden), v=(kvd, cfg.hidden), o=(cfg.hidden, qd),
                      gate=(cfg.inter, cfg.hidden), up=(cfg.inter, cfg.hidden), down=(cfg.hidden, cfg.inter))
        p = {name: proj(name, li, *sh) for name, sh in shapes.items()}
        an = inputs.norm_weights_np(inputs.seed_for(tag, li, "attn_norm"), cfg.hidden)
        fn = inputs.norm_weights_np(inputs.seed_for(tag, li, "ffn_norm"), cfg.hidden)
        qn = inputs.norm_weights_np(inputs.seed_for(tag, li, "q"), cfg.head_dim) if qk_norm else None
        kn = inputs.norm_weights_np(inputs.seed_for(tag, li, "k"), cfg.head_dim) if qk_norm else None
        cu = lambda a: None if a is None else torch.from_numpy(a).cuda()
        dev_layers.append(LayerWeights(p["q"][0], p["k"][0], p["v"][0], p["o"][0], p["gate"][0], p["up"][0],
                                       p["down"][0], cu(an), cu(fn), cu(qn), cu(kn)))
        ref_layers.append(dict(wq=p["q"][1], wk=p["k"][1], wv=p["v"][1], wo=p["o"][1], wg=p["gate"][1],
                               wu=p["up"][1], wd=p["down"][1], attn_norm=an.astype(np.float64),
                               ffn_norm=fn.astype(np.float64)))
        if qk_norm:
            ref_layers[-1].update(q_norm=qn.astype(np.float64), k_norm=kn.astype(np.float64))
    emb = inputs.activations_np(inputs.seed_for(tag, 0, "emb"), (cfg.vocab, cfg.hidden))
    norm = inputs.norm_weights_np(inputs.seed_for(tag, 0, "norm"), cfg.hidden)
    head_dev, head_ref = proj("lm_head", 0, cfg.vocab, cfg.hidden)
    ref = dict(emb=emb.astype(np.float64), layers=ref_layers, norm=norm.astype(np.float64), lm_head=head_ref,
               hq=cfg.n_q_heads, hkv=cfg.n_kv_heads, d=cfg.head_dim, eps=cfg.eps, theta=cfg.theta)
    if cfg.rope_scaling is not None:
        ref["rope_scaling"] = cfg.rope_scaling
    return dev_layers, torch.from_numpy(emb).cuda(), torch.from_numpy(norm).cuda(), head_dev, ref


def _decoder(cfg, tag, max_len, fmts=(O.Q4, B.Q4_G32), fused=True, rope_epi=True, qk_norm=False):
    rope_epi = rope_epi and fused and not qk_norm
    layers, emb, norm, head, ref = _model(cfg, tag, fmts, interleave=rope_epi, qk_norm=qk_norm)
    dec = DenseDecoder(cfg, emb, layers, norm, head, max_len, fused=fused, rope_rows_interleaved=rope_epi)
    assert dec.fused == fused
    kc = np.zeros((cfg.layers, cfg.n_kv_heads, max_len, cfg.head_dim))
    vc = np.zeros_like(kc)
    return dec, ref, kc, vc


TINY = DecoderConfig(hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, inter=512, vocab=1000, layers=2,
                     theta=1e4)


@pytest.mark.parametrize("fused,rope_epi", [(True, True), (True, False), (False, False)])
def test_decode_steps_teacher_forced_tiny(fused, rope_epi):
    """Ten teacher-forced steps: logits at every step, then the whole caches
    (norms and RoPE fused into the q/k/v GEMV; norms fused only; every step
    a launch of its own)."""
    dec, ref, kc, vc = _decoder(TINY, 21, 16, fused=fused, rope_epi=rope_epi)
    for pos, t in enumerate([5, 17, 999, 0, 42, 42, 7, 300, 1, 2]):
        dec.token.fill_(t)
        dec.step(pos)
        want = O.decode_step(ref, t, pos, kc, vc)
        assert rel_err(dec.logits.cpu().numpy(), want) <= GEMV_TOL, pos
    assert rel_err(dec.k_cache.cpu().numpy().astype(np.float64), kc) <= 2e-3
    assert rel_err(dec.v_cache.cpu().numpy().astype(np.float64), vc) <= 2e-3
    assert torch.all(dec.k_cache[:, :, 10:] == 0) and torch.all(dec.v_cache[:, :, 10:] == 0)


@pytest.mark.parametrize("fmts", [(O.Q3, B.Q3_G32), (O.Q6, B.Q6_G32), (O.BF16, B.BF16)])
def test_decode_steps_fused_other_formats(fmts):
    """Norms and RoPE fused into the GEMVs with Q3, Q6 and BF16 weights:
    logits of four teacher-forced steps and the caches against the oracle."""
    dec, ref, kc, vc = _decoder(TINY, 23, 8, fmts=fmts, fused=True, rope_epi=True)
    for pos, t in enumerate([5, 999, 0, 42]):
        dec.token.fill_(t)
        dec.step(pos)
        want = O.decode_step(ref, t, pos, kc, vc)
        assert rel_err(dec.logits.cpu().numpy(), want) <= GEMV_TOL, pos
    assert rel_err(dec.k_cache.cpu().numpy().astype(np.float64), kc) <= 2e-3
    assert rel_err(dec.v_cache.cpu().numpy().astype(np.float64), vc) <= 2e-3


def test_decode_steps_greedy_chain_q8_d128():
    """Greedy generation with the token kept on the device: every sampled id
    is the argmax of that step's logits, and the oracle fed the same ids
    gives the same logits.  head_dim 128, 8 query heads per KV head, Q8."""
    cfg = DecoderConfig(hidden=512, n_q_heads=16, n_kv_heads=2, head_dim=128, inter=1024, vocab=3001, layers=1)
    dec, ref, kc, vc = _decoder(cfg, 22, 32, fmts=(O.Q8, B.Q8_G32))
    dec.token.fill_(3)
    t = 3
    for pos in range(6):
        dec.step(pos)
        logits = dec.logits.cpu().numpy()
        want = O.decode_step(ref, t, pos, kc, vc)
        assert rel_err(logits, want) <= GEMV_TOL, pos
        t = int(dec.token.item())
        assert t == O.greedy_token(logits)


def test_decode_step_qwen3_widths_long_context():
    """Qwen3-0.6B layer widths (hidden 1024, 16 / 8 heads of 128, FFN 3072),
    two layers, a 20000-entry vocabulary, at positions 1000 and 1001 over a
    cache pre-filled with seeded values (the same on both sides)."""
    cfg = DecoderConfig(hidden=1024, n_q_heads=16, n_kv_heads=8, head_dim=128, inter=3072, vocab=20000, layers=2)
    p0 = 1000
    dec, ref, kc, vc = _decoder(cfg, 23, 1024)
    pre_k = inputs.activations_np(inputs.seed_for(23, 0, "cache"), kc.shape)
    pre_v = inputs.activations_np(inputs.seed_for(23, 1, "cache"), kc.shape)
    pre_k[:, :, p0:] = 0
    pre_v[:, :, p0:] = 0
    dec.k_cache.copy_(torch.from_numpy(pre_k))
    dec.v_cache.copy_(torch.from_numpy(pre_v))
    kc[:] = pre_k
    vc[:] = pre_v
    for pos, t in ((p0, 12345), (p0 + 1, 19999)):
        dec.token.fill_(t)
        dec.step(pos)
        assert rel_err(dec.logits.cpu().numpy(), O.decode_step(ref, t, pos, kc, vc)) <= GEMV_TOL, pos


def test_decode_step_graph_replay_matches_eager():
    """A captured step replayed several times (eager work and
    synchronisations between replays) gives the eager step's logits and
    token each time."""
    dec, _, _, _ = _decoder(TINY, 24, 16)
    dec.token.fill_(11)
    dec.step(0)
    dec.token.fill_(11)
    dec.step(1)
    eager_logits, eager_tok = dec.logits.clone(), dec.token.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        dec.token.fill_(11)
        with torch.cuda.graph(g, stream=s):
            dec.step(1)
    torch.cuda.current_stream().wait_stream(s)
    for _ in range(3):
        dec.token.fill_(11)
        dec.logits.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(dec.logits, eager_logits) and torch.equal(dec.token, eager_tok)


# ---------------------------------------------------------------- fp16 outputs

@pytest.mark.parametrize("fmt", [B.Q4_G32, B.Q8_G32, B.Q3_G32])
@pytest.mark.parametrize("n,k", [(65, 96), (3072, 1024), (8192, 3072), (16448, 256)])
def test_gemv_swiglu_f16_is_the_rounded_fp32_output(fmt, n, k):
    w = [B.qm_repack(B.qm_quantise(inputs.weights_dev(inputs.seed_for(31, n, t), (n, k)), fmt), B.LAYOUT_DEVICE)
         for t in ("gate", "up")]
    x = inputs.activations_dev(inputs.seed_for(31, n, "x"), (k,))
    h32 = B.qmatmul_gemv_swiglu(w[0], w[1], x)
    h16 = B.qmatmul_gemv_swiglu(w[0], w[1], x, out=torch.empty(n, dtype=torch.float16, device="cuda"))
    assert torch.equal(h16, h32.half())


@pytest.mark.parametrize("d,hq,hkv", [(64, 32, 8), (128, 16, 8), (128, 24, 8)])
@pytest.mark.parametrize("length", [1, 100, 128, 129, 3000])
def test_attention_decode_f16_is_the_rounded_fp32_output(d, hq, hkv, length):
    max_len = 4096
    q = inputs.activations_dev(inputs.seed_for(32, length, "q"), (hq, d))
    kc = inputs.activations_dev(inputs.seed_for(32, length, "k"), (hkv, max_len, d))
    vc = inputs.activations_dev(inputs.seed_for(32, length, "v"), (hkv, max_len, d))
    o32 = B.qattn_decode(q, kc, vc, length, 1 / math.sqrt(d))
    o16 = B.qattn_decode(q, kc, vc, length, 1 / math.sqrt(d), out=torch.empty((hq, d), dtype=torch.float16,
                                                                              device="cuda"))
    assert torch.equal(o16, o32.half())


# ---------------------------------------------------------------- fused norms

def _norm_inputs(k, tag, with_res):
    rng = np.random.default_rng(tag + k)
    x = (rng.standard_normal(k) * 2).astype(np.float32)
    r = rng.standard_normal(k).astype(np.float32) if with_res else None
    g = inputs.norm_weights_np(tag + k, k)
    n = O.f16(O.rmsnorm(x.astype(np.float64) + (r if with_res else 0.0), g, 1e-6))
    dev = lambda a: None if a is None else torch.from_numpy(a).cuda()
    return dev(x), dev(r), dev(g), n, x, r


@pytest.mark.parametrize("fmt", [(O.Q4, B.Q4_G32), (O.Q8, B.Q8_G32)])
@pytest.mark.parametrize("k,ns", [(256, (64, 32, 32)), (1024, (2048, 1024, 1024)), (1024, (100, 37, 260)),
                                  (3072, (3072, 1024, 1024)), (4096, (16448,)), (2048, (2048, 512, 512))])
@pytest.mark.parametrize("with_res", [False, True])
def test_gemv_grouped_rmsnorm_parity(fmt, k, ns, with_res):
    ofmt, bfmt = fmt
    xd, rd, gd, n, x, r = _norm_inputs(k, 41, with_res)
    ws, refs = [], []
    for i, nn in enumerate(ns):
        w = inputs.weights_np(inputs.seed_for(41, nn, "q", i), (nn, k))
        ws.append(B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), bfmt), B.LAYOUT_DEVICE))
        q, s = O.quantise(w, ofmt)
        refs.append(O.gemv(O.pack(q, ofmt), s, ofmt, n))
    x_out = torch.empty(k, device="cuda")
    ys = B.qmatmul_gemv_grouped_rmsnorm(ws, xd, gd, 1e-6, x_out, residual=rd)
    for y, ref in zip(ys, refs):
        assert rel_err(y.cpu().numpy(), ref) <= GEMV_TOL
    assert np.array_equal(x_out.cpu().numpy(), x + r if with_res else x)
    # the composition of the two separate launches agrees to within fp16 rounding of n
    h = B.qdec_rmsnorm(xd.clone(), gd, 1e-6, residual=rd)
    two = B.qmatmul_gemv_grouped(ws, [h] * len(ws))
    for y, t in zip(ys, two):
        assert rel_err(y.cpu().numpy(), t.cpu().numpy().astype(np.float64)) <= 2e-3


@pytest.mark.parametrize("fmt", [(O.Q4, B.Q4_G32), (O.Q8, B.Q8_G32)])
@pytest.mark.parametrize("n,k", [(65, 96), (3072, 1024), (8192, 3072), (8192, 2048), (16448, 256)])
def test_gemv_swiglu_rmsnorm_parity(fmt, n, k):
    ofmt, bfmt = fmt
    xd, rd, gd, nrm, x, r = _norm_inputs(k, 42, True)
    wg = inputs.weights_np(inputs.seed_for(42, n, "gate"), (n, k))
    wu = inputs.weights_np(inputs.seed_for(42, n, "up"), (n, k))
    dev = [B.qm_repack(B.qm_quantise(torch.from_numpy(w).cuda(), bfmt), B.LAYOUT_DEVICE) for w in (wg, wu)]
    (gq, gs), (uq, us) = O.quantise(wg, ofmt), O.quantise(wu, ofmt)
    ref = O.gemv_swiglu(O.pack(gq, ofmt), gs, O.pack(uq, ofmt), us, ofmt, nrm)
    x_out = torch.empty(k, device="cuda")
    h = B.qmatmul_gemv_swiglu_rmsnorm_f16(dev[0], dev[1], xd, gd, 1e-6, x_out, residual=rd)
    assert rel_err(h.float().cpu().numpy(), ref) <= GEMV_TOL
    assert np.array_equal(x_out.cpu().numpy(), x + r)


@pytest.mark.parametrize("fmt", [B.Q4_G32, B.Q8_G32])
@pytest.mark.parametrize("d,hq,hkv,k", [(64, 4, 2, 256), (128, 16, 8, 1024), (64, 32, 8, 2048), (128, 24, 8, 3072)])
@pytest.mark.parametrize("pos", [0, 5, 1000])
def test_gemv_qkv_rmsnorm_rope_matches_separate_launches(fmt, d, hq, hkv, k, pos):
    """The RoPE epilogue on interleaved rows against the grouped norm GEMV on
    the natural rows followed by qdec_rope_append: caches and q within one
    fp16 ulp (fp32 rotations of the same products), rows other than pos
    untouched, x_out bit for bit."""
    max_len, theta = 1024, 1e6
    xd, rd, gd, _, _, _ = _norm_inputs(k, 43, True)
    w = [inputs.weights_dev(inputs.seed_for(43, k, t), (n, k), sigma=1.0 / math.sqrt(k))
         for t, n in (("q", hq * d), ("k", hkv * d), ("v", hkv * d))]
    plain = [B.qm_repack(B.qm_quantise(a, fmt), B.LAYOUT_DEVICE) for a in w]
    inter = [B.qm_repack(B.qm_quantise(B.rope_interleave_rows(a, n // d, d), fmt), B.LAYOUT_DEVICE)
             for a, n in ((w[0], hq * d), (w[1], hkv * d))] + [plain[2]]
    kc1 = inputs.activations_dev(inputs.seed_for(43, pos, "k"), (hkv, max_len, d))
    vc1 = inputs.activations_dev(inputs.seed_for(43, pos, "v"), (hkv, max_len, d))
    kc2, vc2 = kc1.clone(), vc1.clone()
    xo1, xo2 = torch.empty(k, device="cuda"), torch.empty(k, device="cuda")
    ys = B.qmatmul_gemv_grouped_rmsnorm(plain, xd, gd, 1e-6, xo1, residual=rd)
    q1 = B.qdec_rope_append(ys[0], ys[1], ys[2], pos, theta, kc1, vc1)
    tab = B.qdec_rope_table(max_len, d, theta)
    q2 = torch.empty((hq, d), dtype=torch.float16, device="cuda")
    B.qmatmul_gemv_qkv_rmsnorm_rope(inter, xd, gd, 1e-6, xo2, pos, tab, q2, kc2, vc2, residual=rd)
    assert torch.equal(xo1, xo2)
    for a, b in ((q1, q2), (kc1[:, pos], kc2[:, pos]), (vc1[:, pos], vc2[:, pos])):
        a, b = a.float(), b.float()
        assert torch.all((a - b).abs() <= 2.0 ** -9 * a.abs() + 1e-6 * a.abs().max()), (a - b).abs().max()
    other = torch.ones(max_len, dtype=torch.bool)
    other[pos] = False
    assert torch.equal(kc1[:, other], kc2[:, other]) and torch.equal(vc1[:, other], vc2[:, other])


OTHER_FMTS = [(O.Q2, B.Q2_G32), (O.Q3, B.Q3_G32), (O.Q5, B.Q5_G32), (O.Q6, B.Q6_G32), (O.F16, B.F16),
              (O.BF16, B.BF16)]


@pytest.mark.parametrize("fmt", OTHER_FMTS)
@pytest.mark.parametrize("k,ns", [(1024, (100, 37, 260)), (3072, (3072, 1024, 1024)), (2048, (2048, 512, 512))])
def test_gemv_grouped_rmsnorm_other_formats(fmt, k, ns):
    """Q2/Q3/Q5/Q6/F16/BF16 weights: the normed activation staged in LDS by
    the same workgroups (no lane broadcast), against the oracle."""
    test_gemv_grouped_rmsnorm_parity(fmt, k, ns, True)


@pytest.mark.parametrize("fmt", OTHER_FMTS)
@pytest.mark.parametrize("n,k", [(65, 96), (3072, 1024), (8192, 2048)])
def test_gemv_swiglu_rmsnorm_other_formats(fmt, n, k):
    test_gemv_swiglu_rmsnorm_parity(fmt, n, k)


@pytest.mark.parametrize("fmt", [b for _, b in OTHER_FMTS])
@pytest.mark.parametrize("d,hq,hkv,k", [(64, 4, 2, 256), (128, 24, 8, 3072)])
def test_gemv_qkv_rmsnorm_rope_other_formats(fmt, d, hq, hkv, k):
    test_gemv_qkv_rmsnorm_rope_matches_separate_launches(fmt, d, hq, hkv, k, 5)


@pytest.mark.parametrize("d,theta,scaling", [(64, 5e5, (32, 1, 4, 8192)), (128, 5e5, (32, 1, 4, 8192)),
                                              (64, 1e4, (4, 1, 4, 1000)), (128, 1e6, (8, 2, 3, 4096))])
def test_rope_table_llama3_matches_the_oracle_frequencies(d, theta, scaling):
    """qdec_rope_table_llama3 against cos/sin of p * f_i with the oracle's
    scaled frequencies (every regime of the rule occurs in these shapes)."""
    n = 9000
    t = B.qdec_rope_table_llama3(n, d, theta, scaling).cpu().numpy().astype(np.float64)
    f = O.rope_frequencies(d, theta, scaling)
    w = 2 * np.pi / O.rope_frequencies(d, theta)
    assert (w < scaling[3] / scaling[2]).any() and (w > scaling[3] / scaling[1]).any()
    ang = np.arange(n)[:, None] * f[None, :]
    assert np.abs(t[..., 0] - np.cos(ang)).max() <= 2e-7 and np.abs(t[..., 1] - np.sin(ang)).max() <= 2e-7


@pytest.mark.parametrize("fused,rope_epi,qk_norm", [(True, True, False), (False, False, False), (True, False, True)])
def test_decode_and_prefill_with_llama3_rope(fused, rope_epi, qk_norm):
    """A decoder with the Llama 3 RoPE frequencies (the table from
    qdec_rope_table_llama3 read by every RoPE of the step and of the prompt
    path): a 9-token prompt, then three decode steps, against the oracle's
    token-by-token steps with the same rule."""
    cfg = DecoderConfig(hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, inter=512, vocab=1000, layers=2,
                        theta=5e5, rope_scaling=(32, 1, 4, 64))
    dec, ref, kc, vc = _decoder(cfg, 31, 32, fused=fused, rope_epi=rope_epi, qk_norm=qk_norm)
    toks = [5, 17, 999, 0, 42, 42, 7, 300, 1]
    for p, t in enumerate(toks):
        want = O.decode_step(ref, t, p, kc, vc)
    dec.prefill(torch.tensor(toks, dtype=torch.int32, device="cuda"))
    assert rel_err(dec.logits.cpu().numpy(), want) <= 1e-2
    for p, t in enumerate([3, 4, 5], start=len(toks)):
        dec.token.fill_(t)
        dec.step(p)
        assert rel_err(dec.logits.cpu().numpy(), O.decode_step(ref, t, p, kc, vc)) <= 1e-2, p
    n = len(toks) + 3
    assert rel_err(dec.k_cache[:, :, :n].cpu().numpy().astype(np.float64), kc[:, :, :n]) <= 1e-2
    # the rule matters at these positions: the plain-RoPE oracle disagrees
    plain = dict(ref); plain.pop("rope_scaling")
    kc2, vc2 = np.zeros_like(kc), np.zeros_like(vc)
    for p, t in enumerate(toks + [3, 4, 5]):
        O.decode_step(plain, t, p, kc2, vc2)
    assert rel_err(dec.k_cache[:, :, :n].cpu().numpy().astype(np.float64), kc2[:, :, :n]) > 1e-2


def test_rope_table_matches_the_rotation_angles():
    t = B.qdec_rope_table(300, 64, 5e5).cpu().numpy().astype(np.float64)
    p, i = np.meshgrid(np.arange(300), np.arange(32), indexing="ij")
    ang = p * 5e5 ** (-2.0 * i / 64)
    assert np.abs(t[..., 0] - np.cos(ang)).max() <= 1e-7 and np.abs(t[..., 1] - np.sin(ang)).max() <= 1e-7


# ---------------------------------------------------------------- prompt chunks

def test_prefill_glue_kernels():
    rng = np.random.default_rng(50)
    # embedding rows
    table = inputs.activations_np(51, (300, 64))
    toks = np.array([0, 299, 5, -3, 7], np.int32)
    x = B.qdec_embed_rows(torch.from_numpy(table).cuda(), torch.from_numpy(toks).cuda()).cpu().numpy()
    assert np.array_equal(x[[0, 1, 2, 4]], table[[0, 299, 5, 7]].astype(np.float32)) and np.all(np.isnan(x[3]))
    # heads -> rows
    o = rng.standard_normal((6, 33, 64)).astype(np.float32)
    r = B.qdec_heads_to_rows_f16(torch.from_numpy(o).cuda()).cpu().numpy()
    assert np.array_equal(r, o.transpose(1, 0, 2).reshape(33, 6 * 64).astype(np.float16))
    # swiglu
    g = (rng.standard_normal(5000) * 4).astype(np.float32)
    u = rng.standard_normal(5000).astype(np.float32)
    h = B.qdec_swiglu_f16(torch.from_numpy(g).cuda(), torch.from_numpy(u).cuda()).float().cpu().numpy()
    ref = O.silu(g.astype(np.float64)) * u
    assert np.all(np.abs(h - ref) <= 2.0 ** -10 * np.abs(ref) + 1e-6)


@pytest.mark.parametrize("interleaved", [False, True])
@pytest.mark.parametrize("d,m,p0", [(64, 37, 0), (128, 100, 20)])
def test_rope_append_rows_matches_one_token_at_a_time(interleaved, d, m, p0):
    """Every row r equals qdec_rope_append at position p0 + r (same kernel
    arithmetic), for natural and interleaved projection columns."""
    hq, hkv, max_len, theta = 4, 2, 256, 1e4
    rng = np.random.default_rng(d + m)
    q = torch.from_numpy(rng.standard_normal((m, hq * d)).astype(np.float32)).cuda()
    k = torch.from_numpy(rng.standard_normal((m, hkv * d)).astype(np.float32)).cuda()
    v = torch.from_numpy(rng.standard_normal((m, hkv * d)).astype(np.float32)).cuda()
    kc1 = torch.zeros((hkv, max_len, d), dtype=torch.float16, device="cuda")
    vc1, kc2, vc2 = kc1.clone(), kc1.clone(), kc1.clone()
    qi, ki = q, k
    if interleaved:      # columns of each head in the interleaved order
        perm = lambda t, heads: t.reshape(m, heads, 2, d // 2).transpose(2, 3).reshape(m, heads * d).contiguous()
        qi, ki = perm(q, hq), perm(k, hkv)
    qo = B.qdec_rope_append_rows(qi, ki, v, p0, theta, kc1, vc1, interleaved=interleaved)
    for r in range(m):
        q1 = B.qdec_rope_append(q[r].contiguous(), k[r].contiguous(), v[r].contiguous(), p0 + r, theta, kc2, vc2)
        assert torch.equal(qo[:, r], q1), r
    assert torch.equal(kc1, kc2) and torch.equal(vc1, vc2)
    # with the cache's (cos, sin) table: the same bits
    kc3, vc3 = torch.zeros_like(kc1), torch.zeros_like(vc1)
    tab = B.qdec_rope_table(max_len, d, theta)
    qo3 = B.qdec_rope_append_rows(qi, ki, v, p0, theta, kc3, vc3, interleaved=interleaved, table=tab)
    assert torch.equal(qo3, qo) and torch.equal(kc3, kc1) and torch.equal(vc3, vc1)


@pytest.mark.parametrize("rope_epi", [False, True])
def test_prefill_then_decode_matches_oracle(rope_epi):
    """A prompt of 13 tokens through the prefill path (GEMMs, causal
    attention), then three decode steps: every step's logits and the caches
    against the oracle's token-by-token steps (GEMM tier: fp16 MFMA operands)."""
    dec, ref, kc, vc = _decoder(TINY, 25, 32, rope_epi=rope_epi)
    toks = [5, 17, 999, 0, 42, 42, 7, 300, 1, 2, 64, 65, 998]
    for p, t in enumerate(toks):
        want = O.decode_step(ref, t, p, kc, vc)
    dec.prefill(torch.tensor(toks, dtype=torch.int32, device="cuda"))
    assert rel_err(dec.logits.cpu().numpy(), want) <= 1e-2
    n = len(toks)
    assert rel_err(dec.k_cache[:, :, :n].cpu().numpy().astype(np.float64), kc[:, :, :n]) <= 1e-2
    assert rel_err(dec.v_cache[:, :, :n].cpu().numpy().astype(np.float64), vc[:, :, :n]) <= 1e-2
    for p, t in enumerate([3, 4, 5], start=n):
        dec.token.fill_(t)
        dec.step(p)
        assert rel_err(dec.logits.cpu().numpy(), O.decode_step(ref, t, p, kc, vc)) <= 1e-2, p


def test_prefill_chunks_match_one_chunk():
    """Two chunks (positions 0..19, then 20..44) give the caches and logits
    of one 45-token chunk, to the GEMM tier."""
    cfg = DecoderConfig(hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=128, inter=1024, vocab=2000, layers=2)
    toks = torch.from_numpy(np.random.default_rng(52).integers(0, 2000, 45).astype(np.int32)).cuda()
    a, _, _, _ = _decoder(cfg, 26, 64)
    b, _, _, _ = _decoder(cfg, 26, 64)
    a.prefill(toks)
    b.prefill(toks[:20].contiguous())
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    b.prefill(toks[20:].contiguous(), p0=20)          # chunk buffers reused: nothing allocated
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before
    with pytest.raises(ValueError):
        b.prefill(torch.zeros(b.max_chunk + 1, dtype=torch.int32, device="cuda"))
    assert rel_err(b.logits.cpu().numpy(), a.logits.cpu().numpy().astype(np.float64)) <= 1e-2
    assert rel_err(b.k_cache[:, :, :45].float().cpu().numpy(), a.k_cache[:, :, :45].float().cpu().numpy().astype(np.float64)) <= 1e-2



# ---------------------------------------------------------------- Qwen3 q/k norms

@pytest.mark.parametrize("fused", [True, False])
def test_decode_steps_with_qk_norm(fused):
    """The Qwen3 layer (per-head q/k RMSNorm before RoPE): teacher-forced
    steps against the oracle, head_dim 64 and 128."""
    for cfg, tag in ((TINY, 27), (DecoderConfig(hidden=512, n_q_heads=8, n_kv_heads=4, head_dim=128, inter=768,
                                                 vocab=1500, layers=2), 28)):
        dec, ref, kc, vc = _decoder(cfg, tag, 16, fused=fused, qk_norm=True)
        for pos, t in enumerate([9, 1, 77, 3, 3]):
            dec.token.fill_(t)
            dec.step(pos)
            assert rel_err(dec.logits.cpu().numpy(), O.decode_step(ref, t, pos, kc, vc)) <= GEMV_TOL, (tag, pos)
        assert rel_err(dec.k_cache[:, :, :5].cpu().numpy().astype(np.float64), kc[:, :, :5]) <= 2e-3


def test_prefill_with_qk_norm_matches_oracle():
    dec, ref, kc, vc = _decoder(TINY, 29, 32, qk_norm=True)
    toks = [4, 8, 15, 16, 23, 42, 108, 500, 0]
    for p, t in enumerate(toks):
        want = O.decode_step(ref, t, p, kc, vc)
    dec.prefill(torch.tensor(toks, dtype=torch.int32, device="cuda"))
    assert rel_err(dec.logits.cpu().numpy(), want) <= 1e-2
    assert rel_err(dec.k_cache[:, :, :9].cpu().numpy().astype(np.float64), kc[:, :, :9]) <= 1e-2
