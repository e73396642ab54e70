"""Benchmark of the quantised-matmul hot path on one MI355X.

Default workload (the JSON line's `value`): one decode step of a
Llama-3.2-3B-shaped stack at batch 1 with Q4 group-32 weights -- 28 layers x
{q 3072->3072, k/v 3072->1024, o 3072->3072, gate/up 3072->8192,
down 8192->3072} plus the lm_head 3072->128256, i.e. 197 GEMV calls, each
with its own fp16 activation vector.  All weights (1,807,073,280 bytes of Q4
codes and scales) sit in HBM in the device layout before timing; the 197
calls of a step are captured once in a HIP graph and replayed.

value = Q4 weight bytes streamed per step x steps / elapsed (GB/s).

The line also carries
  roofline:     the dominant GEMV kernel of the step (the projection shape
                with the largest share of the step time): algorithmic weight
                bytes per launch / its mean launch duration, timed with HIP
                events on the launch stream over a graph of all its launches
                of the step back to back; per-shape figures beside it;
  calibration:  achievable rates on this part from torch's own kernels (a
                streaming copy, a hipBLASLt fp16 matmul), as context;
  cpu_baseline: the CPU oracle timed on a bounded sample of the same step
                (whole layers, then a slice of the lm_head), and beside it
                on samples of the prefill GEMM and MoE workloads at M = 128;
  extra:        the other workloads (single 1024x1024 GEMV hot and cold,
                Qwen3-0.6B Q4 and Llama-3.2-3B Q8 decode stacks, Llama-3.2-1B
                prefill GEMM stacks and the Qwen3-30B-A3B MoE layer at M = 128
                / 512 / 2048 (and at M = 512 in the six quantised formats),
                attention and whole-decoder lines), each timed the same way
                (omit with --extra none).

Run: python bench.py [--gpus 1] [--steps K] [--warmup W] [--extra all|none|...]
"""

from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 FLOP/clk (dense fp16)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# --------------------------------------------------------------- helpers

class GemvCall:
    """One pre-marshalled qmatmul_gemv call (descriptor kept alive)."""

    def __init__(self, lib, wd, x, y):
        self.lib, self.wd, self.x, self.y = lib, wd, x, y
        self.desc = wd.c()
        self.ref = ctypes.byref(self.desc)
        self.xp = ctypes.c_void_p(x.data_ptr())
        self.yp = ctypes.c_void_p(y.data_ptr())

    def __call__(self, stream):
        st = self.lib.qmatmul_gemv(self.ref, self.xp, self.yp, stream)
        if st != 0:
            raise RuntimeError(self.lib.qm_last_error().decode())


def build_decode_stack(model, cfg_id, fmt, torch, B, inputs, workloads, want_fp32=False):
    """Quantise + repack every projection of a decode stack on the GPU."""
    lib = B.lib()
    calls, nbytes = [], 0
    for ci, (layer, name, k, n) in enumerate(workloads.stack_calls(model)):
        w = inputs.weights_dev(inputs.seed_for(cfg_id, layer, name), (n, k))
        wd = B.qm_repack(B.qm_quantise(w, fmt), B.LAYOUT_DEVICE)
        del w
        x = inputs.activations_dev(inputs.seed_for(cfg_id, layer, "x", ci), (k,))
        y = torch.empty(n, dtype=torch.float32, device="cuda")
        calls.append(GemvCall(lib, wd, x, y))
        nbytes += workloads.q4_bytes(k, n) if fmt == B.Q4_G32 else workloads.q8_bytes(k, n)
    torch.cuda.synchronize()
    return calls, nbytes


class GroupCall:
    """One pre-marshalled qmatmul_gemv_grouped call."""

    def __init__(self, lib, B, wds, xs, ys):
        self.lib, self.keep = lib, (wds, xs, ys)
        self.args = B.gemv_group_args(wds, xs, ys)

    def __call__(self, stream):
        n, descs, xp, yp = self.args
        st = self.lib.qmatmul_gemv_grouped(n, descs, xp, yp, stream)
        if st != 0:
            raise RuntimeError(self.lib.qm_last_error().decode())


class SwigluCall:
    """One pre-marshalled qmatmul_gemv_swiglu call (gate/up pair, h out)."""

    def __init__(self, lib, wg, wu, x, h):
        self.lib, self.keep = lib, (wg, wu, x, h)
        self.dg, self.du = wg.c(), wu.c()
        self.xp, self.hp = ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(h.data_ptr())

    def __call__(self, stream):
        st = self.lib.qmatmul_gemv_swiglu(ctypes.byref(self.dg), ctypes.byref(self.du), self.xp, self.hp, stream)
        if st != 0:
            raise RuntimeError(self.lib.qm_last_error().decode())


GROUPS = (("q", "k", "v"), ("o",), ("gate", "up"), ("down",))


def build_grouped_stack(model, cfg_id, fmt, torch, B, inputs, workloads, swiglu=False):
    """The same decode step with one launch per group of projections that
    read the same input (q/k/v, o, gate/up, down per layer; the lm_head).
    swiglu: the gate/up pair runs as qmatmul_gemv_swiglu, writing
    silu(gate) * up instead of the two projections."""
    lib = B.lib()
    shapes = {name: (k, n) for name, k, n in model["layer"]}
    calls, nbytes = [], 0
    for layer in range(model["layers"]):
        for gi, group in enumerate(GROUPS):
            k = shapes[group[0]][0]
            x = inputs.activations_dev(inputs.seed_for(cfg_id, layer, "x", 100 + gi), (k,))
            wds, ys = [], []
            for name in group:
                kk, n = shapes[name]
                w = inputs.weights_dev(inputs.seed_for(cfg_id, layer, name), (n, kk))
                wds.append(B.qm_repack(B.qm_quantise(w, fmt), B.LAYOUT_DEVICE))
                del w
                ys.append(torch.empty(n, dtype=torch.float32, device="cuda"))
                nbytes += workloads.q4_bytes(kk, n) if fmt == B.Q4_G32 else workloads.q8_bytes(kk, n)
            if swiglu and group == ("gate", "up"):
                calls.append(SwigluCall(lib, wds[0], wds[1], x, ys[0]))
            else:
                calls.append(GroupCall(lib, B, wds, [x] * len(group), ys))
    k, n = model["lm_head"]
    w = inputs.weights_dev(inputs.seed_for(cfg_id, model["layers"], "lm_head"), (n, k))
    wd = B.qm_repack(B.qm_quantise(w, fmt), B.LAYOUT_DEVICE)
    del w
    x = inputs.activations_dev(inputs.seed_for(cfg_id, model["layers"], "x"), (k,))
    calls.append(GemvCall(lib, wd, x, torch.empty(n, dtype=torch.float32, device="cuda")))
    nbytes += workloads.q4_bytes(k, n) if fmt == B.Q4_G32 else workloads.q8_bytes(k, n)
    torch.cuda.synchronize()
    return calls, nbytes


def capture(torch, fn):
    """Capture fn(stream_ptr) into a graph on a side stream; returns the graph."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for _ in range(2):                       # eager warm-up outside capture
            fn(ctypes.c_void_p(s.cuda_stream))
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn(ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    return g


def time_graph(torch, g, steps, warmup):
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(st)
    for _ in range(steps):
        g.replay()
    e1.record(st)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return e0.elapsed_time(e1) / 1e3, wall      # seconds (events), seconds (wall)


def steady_launch_us(torch, B, call, copies, reps=24, passes=5):
    """Per-launch time of one GEMV run back to back in a graph (reps launches
    cycling over `copies` copies of the weights, so that the bytes of one
    cycle exceed the 256 MB MALL and every launch streams from HBM)."""
    lib = B.lib()
    wd = call.wd
    ws = [wd] + [B.QWeight(wd.format, wd.layout, wd.batch, wd.n, wd.k, wd.qdata.clone(), wd.scales.clone())
                 for _ in range(copies - 1)]
    descs = [w.c() for w in ws]

    def run(s):
        for r in range(reps):
            st = lib.qmatmul_gemv(ctypes.byref(descs[r % copies]), call.xp, call.yp, s)
            if st != 0:
                raise RuntimeError(lib.qm_last_error().decode())
    g = capture(torch, run)
    t, _ = time_graph(torch, g, passes, 1)
    del g, ws
    return t / passes / reps * 1e6


def per_launch_ms(torch, calls, passes=5):
    """Mean duration of each call, timed with an event pair around every
    launch on the launch stream (eager, not captured)."""
    st = torch.cuda.current_stream()
    sp = ctypes.c_void_p(st.cuda_stream)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in calls]
    tot = [0.0] * len(calls)
    for _ in range(passes):
        for c, (a, b) in zip(calls, ev):
            a.record(st)
            c(sp)
            b.record(st)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(ev):
            tot[i] += a.elapsed_time(b)
    return [t / passes for t in tot]


# --------------------------------------------------------- CPU baseline

def host_info():
    """Core count and CPU model of the host, and numpy's BLAS threads."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        blas = 1
    return {"nproc": os.cpu_count(), "cpu_model": model, "blas_threads": blas}


def cpu_baseline(budget_s: float):
    """The CPU oracle on a bounded sample of the headline workload: whole
    layers of the Llama-3.2-3B Q4 decode step (all seven GEMVs of a layer),
    then rows of the lm_head, until about budget_s seconds of oracle time.
    Only the oracle's GEMV is timed; its inputs (the oracle's own
    quantisation and packing of the same seeded weights) are prepared
    beforehand on a thread pool and are not timed."""
    import concurrent.futures as cf
    from oracle import qmatmul_oracle as O
    from paper_2607_00501_amd import inputs, workloads
    info = host_info()
    model = workloads.LLAMA32_3B

    def prep(item):
        layer, name, ci, k, n = item
        w = inputs.weights_np(inputs.seed_for(2, layer, name), (n, k))
        q, s = O.quantise(w, O.Q4)
        return O.pack(q, O.Q4), s, inputs.activations_np(inputs.seed_for(2, layer, "x", ci), (k,)), k, n

    # about 2.3 s of oracle time per layer (56.6 MB at ~0.025 GB/s)
    layers = max(1, min(model["layers"], int(budget_s * 0.6 / 2.3)))
    items = [(l, name, ci, k, n) for l in range(layers) for ci, (name, k, n) in enumerate(model["layer"])]
    k, n_full = model["lm_head"]
    rows = min(n_full, 32768)
    with cf.ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1))) as ex:
        prepared = list(ex.map(prep, items + [(model["layers"], "lm_head", 0, k, rows)]))
    spent, nbytes = 0.0, 0
    for qb, sc, x, kk, nn in prepared:
        t0 = time.perf_counter()
        O.gemv(qb, sc, O.Q4, x)
        spent += time.perf_counter() - t0
        nbytes += workloads.q4_bytes(kk, nn)
    return {"value": round(nbytes / spent / 1e9, 4), "unit": "GB/s", "cores": info["blas_threads"],
            "kind": "oracle", **info,
            "sample": f"{len(items)} GEMVs (layers 0-{layers - 1}, all 7 projections) + lm_head rows "
                      f"0-{rows - 1} of the Llama-3.2-3B Q4 decode step; {nbytes} weight bytes in "
                      f"{spent:.2f} s of oracle time (numpy: canonical codes dequantised, fp64 products "
                      f"and sums; the fp64 matrix-vector product on BLAS threads={info['blas_threads']}, "
                      f"the dequantisation on one thread)",
            "other_workloads": cpu_baseline_gemm_moe()}


def cpu_baseline_gemm_moe():
    """The oracle on the other workloads (reported beside the headline's
    baseline): the single 1024 x 1024 GEMV on one thread; one Llama-3.2-1B
    layer's seven GEMMs at M = 128; the Qwen3-30B-A3B MoE layer at M = 128
    routed and bucketed in full, with the FFNs of its first 16 experts'
    buckets.  The oracle's own quantisation and packing is prepared untimed,
    as above."""
    from oracle import qmatmul_oracle as O
    from paper_2607_00501_amd import inputs, workloads
    out = {}
    # The single 1024 x 1024 Q4 GEMV on one thread (median of 5 calls).
    q, sc = O.quantise(inputs.weights_np(inputs.seed_for(0, 0, "q"), (1024, 1024)), O.Q4)
    qb, xv = O.pack(q, O.Q4), inputs.activations_np(inputs.seed_for(0, 0, "x"), (1024,))
    try:
        from threadpoolctl import threadpool_limits
        limit = threadpool_limits(1)
    except Exception:
        limit = None
    ts = []
    for _ in range(5):
        t0 = time.perf_counter()
        O.gemv(qb, sc, O.Q4, xv)
        ts.append(time.perf_counter() - t0)
    if limit is not None:
        limit.unregister()
    t1 = sorted(ts)[2]
    out["single_gemv_1024x1024_q4"] = {"value": round(workloads.q4_bytes(1024, 1024) / t1 / 1e9, 4), "unit": "GB/s",
                                       "threads": 1, "sample": f"the whole GEMV, median of 5 calls ({t1 * 1e3:.2f} ms)"}
    m = 128
    prepared = []
    for name, k, n in workloads.LLAMA32_1B_LAYER:
        q, sc = O.quantise(inputs.weights_np(inputs.seed_for(3, 0, name), (n, k)), O.Q4)
        prepared.append((O.pack(q, O.Q4), sc, inputs.activations_np(inputs.seed_for(3, m, "x"), (m, k)), k, n))
    t0 = time.perf_counter()
    flops = 0
    for qb, sc, x, k, n in prepared:
        O.gemm(qb, sc, O.Q4, x)
        flops += 2 * m * n * k
    dt = time.perf_counter() - t0
    out["llama3.2-1b_prefill_m128"] = {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s",
                                       "sample": f"one layer's 7 GEMMs at M = 128 ({flops} FLOP in {dt:.2f} s)"}
    cfg = workloads.QWEN3_30B_A3B_MOE
    E, K, H, I = cfg["experts"], cfg["top_k"], cfg["hidden"], cfg["inter"]
    sample = 16
    x = inputs.activations_np(inputs.seed_for(4, m, "x"), (m, H)).astype(np.float64)
    lg = inputs.logits_np(inputs.seed_for(4, m, "logits"), (m, E))
    packed = []
    for e in range(sample):
        ws = []
        for t, sh in (("gate", (I, H)), ("up", (I, H)), ("down", (H, I))):
            q, sc = O.quantise(inputs.weights_np(inputs.seed_for(4, e, t), sh), O.Q4)
            ws.append((O.pack(q, O.Q4), sc))
        packed.append(ws)
    t0 = time.perf_counter()
    ids, gates = O.moe_route(lg, K)
    counts, offsets, sorted_assign = O.moe_bucket(ids, E)
    rows_done = 0
    for e in range(sample):
        rows = sorted_assign[offsets[e]:offsets[e + 1]]
        wg, wu, wd = (O.dequantise(qb, sc, O.Q4) for qb, sc in packed[e])
        O.expert_ffn(x[rows // K], wg, wu, wd)
        rows_done += rows.size
    dt = time.perf_counter() - t0
    flops = 2 * rows_done * 3 * H * I
    out["qwen3-30b-a3b_moe_m128"] = {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s",
                                     "sample": f"route + bucket of all {m} tokens, FFNs of experts 0-{sample - 1} "
                                               f"({rows_done} assignments, {flops} FLOP in {dt:.2f} s)"}
    return out


# ------------------------------------------------------------ extras

def extra_workloads(torch, B, inputs, workloads, steps, warmup, which="all"):
    out = {}
    lib = B.lib()
    if which in ("all", "tg"):
        out.update(extra_tg(torch, B, inputs, workloads, steps, warmup, lib))
    if which in ("all", "decode"):
        out.update(extra_decode(torch, B, inputs, workloads, steps, warmup, lib))
    if which == "qwen-stack":                 # the Qwen3-0.6B 197-call stack alone (for kernel traces)
        out.update(extra_qwen_stack(torch, B, inputs, workloads, steps, warmup))
    if which in ("all", "prefill"):
        out.update(extra_prefill(torch, B, inputs, workloads, steps, warmup, lib))
    if which in ("all", "moe"):
        out.update(extra_moe(torch, B, inputs, workloads, steps, warmup, lib))
    return out


def build_decoder(model: dict, cfg_id: int, fmt, max_len, torch, B, inputs, qk_norm: bool = False):
    """A dense decoder of the model's geometry with seeded synthetic weights
    (projections quantised on the device), as DenseDecoder."""
    from paper_2607_00501_amd.decoder import DecoderConfig, DenseDecoder, LayerWeights
    cfg = DecoderConfig(**{k: v for k, v in model.items() if k != "name"})
    qd, kvd = cfg.n_q_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim

    def proj(name, li, n, k):
        w = inputs.weights_dev(inputs.seed_for(cfg_id, li, name), (n, k))
        if name in ("q", "k") and not qk_norm:   # row order of the q/k/v GEMV's RoPE epilogue
            w = B.rope_interleave_rows(w, n // cfg.head_dim, cfg.head_dim)
        q = B.qm_repack(B.qm_quantise(w, fmt), B.LAYOUT_DEVICE)
        del w
        return q

    def gain(name, li):
        return torch.from_numpy(inputs.norm_weights_np(inputs.seed_for(cfg_id, li, name), cfg.hidden)).cuda()

    def hgain(name, li):
        return torch.from_numpy(inputs.norm_weights_np(inputs.seed_for(cfg_id, li, name), cfg.head_dim)).cuda()

    layers = []
    for li in range(cfg.layers):
        layers.append(LayerWeights(proj("q", li, qd, cfg.hidden), proj("k", li, kvd, cfg.hidden),
                                   proj("v", li, kvd, cfg.hidden), proj("o", li, cfg.hidden, qd),
                                   proj("gate", li, cfg.inter, cfg.hidden), proj("up", li, cfg.inter, cfg.hidden),
                                   proj("down", li, cfg.hidden, cfg.inter), gain("attn_norm", li),
                                   gain("ffn_norm", li),
                                   *((hgain("q", li), hgain("k", li)) if qk_norm else ())))
    emb = inputs.activations_dev(inputs.seed_for(cfg_id, 0, "emb"), (cfg.vocab, cfg.hidden))
    head = proj("lm_head", 0, cfg.vocab, cfg.hidden)
    torch.cuda.synchronize()
    return DenseDecoder(cfg, emb, layers, gain("norm", 0), head, max_len, rope_rows_interleaved=not qk_norm)


def tg_tokens_per_s(torch, dec, tokens: int, reps: int):
    """tg-N: N greedy decode steps from an empty cache (positions 0 .. N-1),
    the sampled token fed back on the device, all N steps captured in one
    graph (no host synchronisation between tokens).  Returns (tokens/s,
    replay seconds)."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        dec.token.fill_(1)
        dec.step(0)                                   # eager warm-up
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for pos in range(tokens):
            dec.step(pos)
    torch.cuda.synchronize()
    dec.token.fill_(1)
    t, _ = time_graph(torch, g, reps, 1)
    del g
    return tokens * reps / t, t / reps


def extra_tg(torch, B, inputs, workloads, steps, warmup, lib):
    out = {}
    # End-to-end decode, tg128 (Sec. 4.1): every kernel of a token (embedding,
    # norms, projections, RoPE and cache append, attention, SwiGLU, LM head,
    # greedy sampling): 5 launches per layer (the norms run inside the q/k/v
    # and gate/up GEMVs, RoPE and the cache append in the q/k/v GEMV's
    # epilogue; attention is one launch for caches of up to 128 rows) + 5.
    for model, cfg_id in ((workloads.QWEN3_06B_DECODER, 1), (workloads.LLAMA32_1B_DECODER, 3),
                          (workloads.LLAMA32_3B_DECODER, 2)):
        dec = build_decoder(model, cfg_id, B.Q4_G32, 640, torch, B, inputs)
        tps, t = tg_tokens_per_s(torch, dec, 128, 3)
        key = model["name"] + "_tg128_q4"
        out[key] = {"tokens_per_s": round(tps, 1), "ms_per_token": round(1e3 / tps, 4),
                    "launches_per_token": 5 * model["layers"] + 5, "ms_per_128_tokens": round(t * 1e3, 3)}
        log(f"{key}: {out[key]}")
        # pp512: a 512-token prompt in one chunk (prefill GEMMs, causal
        # attention, the last token's logits and greedy id), one graph
        toks = torch.from_numpy(inputs.np.random.default_rng(cfg_id).integers(
            0, model["vocab"], 512).astype(inputs.np.int32)).cuda()
        dec.prefill(toks)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            dec.prefill(toks)
        t, _ = time_graph(torch, g, 5, 1)
        key = model["name"] + "_pp512_q4"
        out[key] = {"tokens_per_s": round(512 * 5 / t, 1), "ms_per_prompt": round(t / 5 * 1e3, 3)}
        log(f"{key}: {out[key]}")
        del g
        if model is workloads.QWEN3_06B_DECODER:
            # the Qwen3 layer proper: per-head q/k norms before RoPE (in the
            # RoPE kernel, so one launch more per layer than the epilogue path)
            del dec
            dec = build_decoder(model, cfg_id, B.Q4_G32, 640, torch, B, inputs, qk_norm=True)
            tps, t = tg_tokens_per_s(torch, dec, 128, 3)
            key = model["name"] + "_qknorm_tg128_q4"
            out[key] = {"tokens_per_s": round(tps, 1), "ms_per_token": round(1e3 / tps, 4),
                        "launches_per_token": 6 * model["layers"] + 5, "ms_per_128_tokens": round(t * 1e3, 3)}
            log(f"{key}: {out[key]}")
        del dec
        torch.cuda.empty_cache()

    return out


def extra_qwen_stack(torch, B, inputs, workloads, steps, warmup):
    """The Qwen3-0.6B Q4 decode stack: 197 GEMV calls, 335 MB per token."""
    out = {}
    calls, nbytes = build_decode_stack(workloads.QWEN3_06B, 1, B.Q4_G32, torch, B, inputs, workloads)
    g = capture(torch, lambda s: [c(s) for c in calls])
    t, _ = time_graph(torch, g, steps, warmup)
    kh, nh = workloads.QWEN3_06B["lm_head"]
    head_bytes = workloads.q4_bytes(kh, nh)
    head_us = steady_launch_us(torch, B, calls[-1], copies=4, reps=12)
    out["qwen3-0.6b_decode_q4"] = {"tokens_per_s": round(steps / t, 2), "ms_per_token": round(t / steps * 1e3, 4),
                                   "weight_GBps": round(nbytes * steps / t / 1e9, 2),
                                   "frac_hbm_peak": round(nbytes * steps / t / 1e9 / HBM_PEAK_GBS, 4),
                                   "lm_head_steady_us": round(head_us, 3),
                                   "lm_head_steady_GBps": round(head_bytes / head_us / 1e3, 2),
                                   "lm_head_steady_frac": round(head_bytes / head_us / 1e3 / HBM_PEAK_GBS, 4)}
    log(f"qwen3 q4 stack: {out['qwen3-0.6b_decode_q4']}")
    del g, calls
    return out


def extra_decode(torch, B, inputs, workloads, steps, warmup, lib):
    out = {}

    # single Q4 GEMV 1024 x 1024
    cfg = workloads.SINGLE_GEMV
    w = inputs.weights_dev(inputs.seed_for(0, 0, "q"), (cfg["n"], cfg["k"]))
    wd = B.qm_repack(B.qm_quantise(w, B.Q4_G32), B.LAYOUT_DEVICE)
    x = inputs.activations_dev(inputs.seed_for(0, 0, "x"), (cfg["k"],))
    y = torch.empty(cfg["n"], device="cuda")
    call = GemvCall(lib, wd, x, y)
    reps = 100
    g = capture(torch, lambda s: [call(s) for _ in range(reps)])
    t, _ = time_graph(torch, g, max(steps // 5, 5), warmup)
    us = t / (max(steps // 5, 5) * reps) * 1e6
    ms = per_launch_ms(torch, [call], passes=20)[0]
    # cold: 1024 distinct copies of the weights (604 MB per cycle, beyond the
    # L2s and the 256 MB MALL), one launch per copy back to back
    copies = 1024
    qs = torch.stack([wd.qdata] * copies)
    ss = torch.stack([wd.scales] * copies)
    cold_descs = [B.QWeight(wd.format, wd.layout, 1, wd.n, wd.k, qs[i], ss[i]).c() for i in range(copies)]

    def run_cold(st):
        for d in cold_descs:
            rc = lib.qmatmul_gemv(ctypes.byref(d), call.xp, call.yp, st)
            if rc != 0:
                raise RuntimeError(lib.qm_last_error().decode())
    gc = capture(torch, run_cold)
    tc, _ = time_graph(torch, gc, 3, 1)
    us_cold = tc / 3 / copies * 1e6
    wb = workloads.q4_bytes(1024, 1024)
    out["single_gemv_1024x1024_q4"] = {"us_per_call_graph_hot": round(us, 3), "us_per_launch_events": round(ms * 1e3, 3),
                                       "weight_GBps_graph_hot": round(wb / us / 1e3, 2),
                                       "us_per_call_graph_cold": round(us_cold, 3),
                                       "weight_GBps_graph_cold": round(wb / us_cold / 1e3, 2),
                                       "note": "hot: one weight buffer, L2/MALL resident (not HBM); cold: 1024 copies"}
    log(f"config single gemv: {out['single_gemv_1024x1024_q4']}")
    del g, gc, qs, ss, cold_descs

    out.update(extra_qwen_stack(torch, B, inputs, workloads, steps, warmup))
    torch.cuda.empty_cache()

    # Grouped dispatch (qmatmul_gemv_grouped): the Qwen3-0.6B and Llama-3.2-3B
    # Q4 steps with q/k/v and gate/up each in one launch (113 launches/token);
    # and the same with gate/up as the fused SwiGLU pair.
    for model, cfg_id, tag in ((workloads.QWEN3_06B, 1, "qwen3-0.6b"), (workloads.LLAMA32_3B, 2, "llama3.2-3b")):
        for swiglu, key in ((False, "grouped_dispatch"), (True, "grouped_swiglu")):
            calls, nbytes = build_grouped_stack(model, cfg_id, B.Q4_G32, torch, B, inputs, workloads, swiglu)
            g = capture(torch, lambda s: [c(s) for c in calls])
            t, _ = time_graph(torch, g, steps, warmup)
            out[f"{tag}_decode_q4_{key}"] = {
                "launches_per_token": len(calls), "tokens_per_s": round(steps / t, 2),
                "ms_per_token": round(t / steps * 1e3, 4), "weight_GBps": round(nbytes * steps / t / 1e9, 2),
                "frac_hbm_peak": round(nbytes * steps / t / 1e9 / HBM_PEAK_GBS, 4)}
            log(f"{tag} {key}: {out[f'{tag}_decode_q4_{key}']}")
            del g, calls
            torch.cuda.empty_cache()

    # Llama-3.2-3B decode stack with Q8 weights (the Q4 stack is the headline)
    for fmt, tag in ((B.Q8_G32, "q8"),):
        calls, nbytes = build_decode_stack(workloads.LLAMA32_3B, 2, fmt, torch, B, inputs, workloads)
        g = capture(torch, lambda s: [c(s) for c in calls])
        t, _ = time_graph(torch, g, steps, warmup)
        per = per_launch_ms(torch, calls, passes=3)
        head_ms = per[-1]
        kh, nh = workloads.LLAMA32_3B["lm_head"]
        head_bytes = workloads.q4_bytes(kh, nh) if fmt == B.Q4_G32 else workloads.q8_bytes(kh, nh)
        head_us = steady_launch_us(torch, B, calls[-1], copies=2 if fmt == B.Q4_G32 else 1, reps=12)
        out[f"llama3.2-3b_decode_{tag}"] = {
            "tokens_per_s": round(steps / t, 2), "ms_per_token": round(t / steps * 1e3, 4),
            "weight_GBps": round(nbytes * steps / t / 1e9, 2),
            "frac_hbm_peak": round(nbytes * steps / t / 1e9 / HBM_PEAK_GBS, 4),
            "lm_head_GBps_events": round(head_bytes / (head_ms * 1e-3) / 1e9, 2),
            "lm_head_frac_hbm_peak": round(head_bytes / (head_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "lm_head_steady_us": round(head_us, 3),
            "lm_head_steady_GBps": round(head_bytes / head_us / 1e3, 2),
            "lm_head_steady_frac": round(head_bytes / head_us / 1e3 / HBM_PEAK_GBS, 4)}
        log(f"llama3b {tag}: {out[f'llama3.2-3b_decode_{tag}']}")
        del g, calls
        torch.cuda.empty_cache()

    # The Llama-3.2-3B lm_head (3072 -> 128256) in every weight format, back
    # to back over enough weight copies to stream from HBM every launch.
    call = None
    fm = {}
    for fmt in (B.Q2_G32, B.Q3_G32, B.Q4_G32, B.Q5_G32, B.Q6_G32, B.Q8_G32, B.F16, B.BF16):
        kh, nh = workloads.LLAMA32_3B["lm_head"]
        w = inputs.weights_dev(inputs.seed_for(2, 28, "lm_head"), (nh, kh))
        wd = B.qm_repack(B.qm_quantise(w, fmt), B.LAYOUT_DEVICE)
        del w
        x = inputs.activations_dev(inputs.seed_for(2, 28, "x"), (kh,))
        call = GemvCall(lib, wd, x, torch.empty(nh, dtype=torch.float32, device="cuda"))
        nbytes = workloads.weight_bytes(fmt, kh, nh)
        copies = max(1, -(-600_000_000 // nbytes))
        us = steady_launch_us(torch, B, call, copies=copies, reps=max(12, 2 * copies))
        fm[workloads.FORMAT_NAMES[fmt]] = {"weight_MB": round(nbytes / 1e6, 1), "us": round(us, 3),
                                           "GBps": round(nbytes / us / 1e3, 1),
                                           "frac_hbm_peak": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4)}
        del call, wd
        torch.cuda.empty_cache()
    out["llama3.2-3b_lm_head_by_format"] = fm
    log(f"lm_head by format: {fm}")

    # Decode attention over the KV cache (one layer, one token): Qwen3-0.6B
    # (16 query / 8 KV heads) and Llama-3.2-3B (24 / 8), head_dim 128, cycling
    # over enough cache copies that every call streams K and V from HBM.
    att = {}
    for tag, hq, hkv in (("qwen3-0.6b", 16, 8), ("llama3.2-3b", 24, 8)):
        for length in (1024, 4096, 16384, 65536):
            d = 128
            kv_bytes = 2 * hkv * length * d * 2
            copies = max(1, -(-600_000_000 // kv_bytes))
            g = torch.Generator(device="cuda").manual_seed(length)
            q = torch.randn((hq, d), generator=g, device="cuda").half()
            ks = [torch.randn((hkv, length, d), generator=g, device="cuda").half() for _ in range(copies)]
            vs = [torch.randn((hkv, length, d), generator=g, device="cuda").half() for _ in range(copies)]
            o = torch.empty((hq, d), dtype=torch.float32, device="cuda")
            ws = torch.empty(B.qattn_decode_workspace_bytes(hq, d), dtype=torch.uint8, device="cuda")
            reps = max(8, 2 * copies)

            def run(st, ks=ks, vs=vs, q=q, o=o, ws=ws, hq=hq, hkv=hkv, length=length, reps=reps):
                for r in range(reps):
                    rc = lib.qattn_decode(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(ks[r % len(ks)].data_ptr()),
                                          ctypes.c_void_p(vs[r % len(vs)].data_ptr()), hq, hkv, 128, length, length,
                                          ctypes.c_float(1.0 / 128 ** 0.5), ctypes.c_void_p(o.data_ptr()),
                                          ctypes.c_void_p(ws.data_ptr()), ws.numel(), st)
                    if rc != 0:
                        raise RuntimeError(lib.qm_last_error().decode())
            gr = capture(torch, run)
            t, _ = time_graph(torch, gr, 5, 1)
            us = t / 5 / reps * 1e6
            att[f"{tag}_len{length}"] = {"us_per_call": round(us, 3), "kv_MB": round(kv_bytes / 1e6, 2),
                                         "GBps": round(kv_bytes / us / 1e3, 1),
                                         "frac_hbm_peak": round(kv_bytes / us / 1e3 / HBM_PEAK_GBS, 4)}
            del gr, ks, vs
            torch.cuda.empty_cache()
    out["decode_attention"] = att
    log(f"decode attention: {att}")
    return out


def extra_prefill(torch, B, inputs, workloads, steps, warmup, lib):
    out = {}
    # Llama-3.2-1B prefill GEMM stacks: Q4 with one launch per GEMM and with
    # grouped dispatch; Q8 weights with grouped dispatch.
    model = workloads.LLAMA32_1B_PREFILL
    reps = max(steps // 2, 5)
    for fmt, tag in ((B.Q4_G32, ""), (B.Q8_G32, "_q8")):
        wds = []
        for layer in range(model["layers"]):
            for name, k, n in model["layer"]:
                w = inputs.weights_dev(inputs.seed_for(3, layer, name), (n, k))
                wds.append((B.qm_repack(B.qm_quantise(w, fmt), B.LAYOUT_DEVICE), k, n))
                del w
        for m in model["m_sweep"]:
            xs = {k: inputs.activations_dev(inputs.seed_for(3, 0, "x", k), (m, k)) for k in {k for _, k, _ in wds}}
            ys = [torch.empty((m, n), device="cuda") for _, _, n in wds]
            flops = 2.0 * m * sum(k * n for _, k, n in wds)
            if fmt == B.Q4_G32:
                descs = [wd.c() for wd, _, _ in wds]

                def run(s, xs=xs, ys=ys, descs=descs, m=m):
                    for d, (wd, k, n), yv in zip(descs, wds, ys):
                        st = lib.qmatmul_gemm(ctypes.byref(d), ctypes.c_void_p(xs[k].data_ptr()), m,
                                              ctypes.c_void_p(yv.data_ptr()), s)
                        if st:
                            raise RuntimeError(lib.qm_last_error().decode())
                g = capture(torch, run)
                t, _ = time_graph(torch, g, reps, warmup)
                tf = flops * reps / t / 1e12
                out[f"llama3.2-1b_prefill_m{m}"] = {"tokens_per_s": round(m * reps / t, 1),
                                                    "stack_TFLOPs": round(tf, 2),
                                                    "frac_mfma_peak": round(tf / MFMA_F16_PEAK_TFLOPS, 4)}
                log(f"prefill m={m}: {out[f'llama3.2-1b_prefill_m{m}']}")
                del g

            # Grouped dispatch (qmatmul_gemm_grouped): q/k/v and gate/up of a
            # layer each in one launch (64 launches for the 16 layers).
            per_layer = len(model["layer"])
            names = [name for name, _, _ in model["layer"]]
            calls = []
            for layer in range(model["layers"]):
                base = layer * per_layer
                for group in GROUPS:
                    idx = [base + names.index(nm) for nm in group]
                    k = wds[idx[0]][1]
                    n_, descs_g, yp = B.gemm_group_args([wds[i][0] for i in idx], [ys[i] for i in idx])
                    calls.append((n_, descs_g, ctypes.c_void_p(xs[k].data_ptr()), yp))

            def run_g(s, calls=calls, m=m):
                for n_, descs_g, xp, yp in calls:
                    st = lib.qmatmul_gemm_grouped(n_, descs_g, xp, m, yp, s)
                    if st:
                        raise RuntimeError(lib.qm_last_error().decode())
            g = capture(torch, run_g)
            t, _ = time_graph(torch, g, reps, warmup)
            tf = flops * reps / t / 1e12
            key = f"llama3.2-1b_prefill{tag}_m{m}_grouped_dispatch"
            out[key] = {"launches_per_stack": len(calls), "tokens_per_s": round(m * reps / t, 1),
                        "stack_TFLOPs": round(tf, 2), "frac_mfma_peak": round(tf / MFMA_F16_PEAK_TFLOPS, 4)}
            log(f"prefill{tag} m={m} grouped: {out[key]}")
            del g, calls, ys, xs
        del wds
        torch.cuda.empty_cache()

    # The prefill GEMM in every weight format: the Llama-3.2-1B gate
    # projection 2048 -> 8192 at M = 512 and 2048, 16 distinct weight copies
    # per graph (134 MB of F16 / BF16 weights, beyond the MALL), back to back.
    fmts = {"q2": B.Q2_G32, "q3": B.Q3_G32, "q4": B.Q4_G32, "q5": B.Q5_G32, "q6": B.Q6_G32, "q8": B.Q8_G32,
            "f16": B.F16, "bf16": B.BF16}
    k, n, copies = 2048, 8192, 16
    by_fmt = {}
    w = inputs.weights_dev(inputs.seed_for(3, 0, "gate"), (n, k))
    for name, fmt in fmts.items():
        wd = B.qm_repack(B.qm_quantise(w, fmt), B.LAYOUT_DEVICE)
        ws = [B.QWeight(wd.format, wd.layout, 1, n, k, wd.qdata.clone(),
                        None if wd.scales is None else wd.scales.clone()) for _ in range(copies)]
        descs = [wi.c() for wi in ws]
        for m in (512, 2048):
            x = inputs.activations_dev(inputs.seed_for(3, m, "x"), (m, k))
            ys = [torch.empty((m, n), device="cuda") for _ in range(copies)]

            def run_f(s, x=x, ys=ys, descs=descs, m=m):
                for d, yv in zip(descs, ys):
                    st = lib.qmatmul_gemm(ctypes.byref(d), ctypes.c_void_p(x.data_ptr()), m,
                                          ctypes.c_void_p(yv.data_ptr()), s)
                    if st:
                        raise RuntimeError(lib.qm_last_error().decode())
            g = capture(torch, run_f)
            t, _ = time_graph(torch, g, reps, warmup)
            us = t / reps / copies * 1e6
            tf = 2.0 * m * n * k / us / 1e6
            by_fmt[f"{name}_m{m}"] = {"us": round(us, 2), "TFLOPs": round(tf, 1),
                                      "frac_mfma_peak": round(tf / MFMA_F16_PEAK_TFLOPS, 4)}
            del g, ys, x
        del ws, descs, wd
        torch.cuda.empty_cache()
    del w
    out["llama3.2-1b_gate_gemm_by_format"] = by_fmt
    log(f"gemm by format: {by_fmt}")

    # Causal prefill attention of one layer (qattn_prefill): Llama-3.2-1B
    # (32 query / 8 KV heads, head_dim 64) and Qwen3-0.6B (16 / 8, head_dim
    # 128); FLOPs 2 * 2 * D * Hq * M(M+1)/2 (the causal half of Q K^T and P V).
    att = {}
    for tag, hq, hkv, d in (("llama3.2-1b", 32, 8, 64), ("qwen3-0.6b", 16, 8, 128)):
        for m in model["m_sweep"]:
            g = torch.Generator(device="cuda").manual_seed(m)
            q = torch.randn((hq, m, d), generator=g, device="cuda").half()
            kc = torch.randn((hkv, m, d), generator=g, device="cuda").half()
            vc = torch.randn((hkv, m, d), generator=g, device="cuda").half()
            o = torch.empty((hq, m, d), dtype=torch.float32, device="cuda")
            nws = B.qattn_prefill_workspace_bytes(hq, d, m, 0)
            aws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")

            def run_a(st, q=q, kc=kc, vc=vc, o=o, hq=hq, hkv=hkv, d=d, m=m, aws=aws):
                for _ in range(10):
                    rc = lib.qattn_prefill(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(kc.data_ptr()),
                                           ctypes.c_void_p(vc.data_ptr()), hq, hkv, d, m, 0, m,
                                           ctypes.c_float(d ** -0.5), ctypes.c_void_p(o.data_ptr()),
                                           ctypes.c_void_p(aws.data_ptr()), aws.numel(), st)
                    if rc:
                        raise RuntimeError(lib.qm_last_error().decode())
            gr = capture(torch, run_a)
            t, _ = time_graph(torch, gr, reps, warmup)
            us = t / reps / 10 * 1e6
            flops = 2.0 * 2.0 * d * hq * m * (m + 1) / 2
            att[f"{tag}_m{m}"] = {"us": round(us, 2), "TFLOPs": round(flops / us / 1e6, 1),
                                  "frac_mfma_peak": round(flops / us / 1e6 / MFMA_F16_PEAK_TFLOPS, 4),
                                  "workspace_MB": round(nws / 1e6, 2)}
            del gr
    # A prompt chunk far into the cache (Qwen3-0.6B heads, 128 rows at
    # position 32,768): its 16 query tiles split over key ranges, against
    # the unsplit single launch.
    hq, hkv, d, m, p0 = 16, 8, 128, 128, 32768
    g = torch.Generator(device="cuda").manual_seed(3)
    q = torch.randn((hq, m, d), generator=g, device="cuda").half()
    kc = torch.randn((hkv, p0 + m, d), generator=g, device="cuda").half()
    vc = torch.randn((hkv, p0 + m, d), generator=g, device="cuda").half()
    o = torch.empty((hq, m, d), dtype=torch.float32, device="cuda")
    nws = B.qattn_prefill_workspace_bytes(hq, d, m, p0)
    aws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")
    chunk = {}
    for mode in ("split", "unsplit"):
        def run_c(st, mode=mode):
            for _ in range(10):
                wp = ctypes.c_void_p(aws.data_ptr()) if mode == "split" else None
                rc = lib.qattn_prefill(ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(kc.data_ptr()),
                                       ctypes.c_void_p(vc.data_ptr()), hq, hkv, d, m, p0, p0 + m,
                                       ctypes.c_float(d ** -0.5), ctypes.c_void_p(o.data_ptr()), wp,
                                       aws.numel() if mode == "split" else 0, st)
                if rc:
                    raise RuntimeError(lib.qm_last_error().decode())
        gr = capture(torch, run_c)
        t, _ = time_graph(torch, gr, reps, warmup)
        us = t / reps / 10 * 1e6
        flops = 2.0 * 2.0 * d * hq * m * (p0 + (m + 1) / 2)
        chunk[mode] = {"us": round(us, 2), "TFLOPs": round(flops / us / 1e6, 1),
                       "kv_GBps": round(2 * hkv * (p0 + m) * d * 2 / us / 1e3, 1)}
        del gr
    att["qwen3-0.6b_m128_at_32768"] = chunk
    out["prefill_attention"] = att
    log(f"prefill attention: {att}")
    return out


def extra_moe(torch, B, inputs, workloads, steps, warmup, lib):
    out = {}
    # Qwen3-30B-A3B MoE layer
    cfg = workloads.QWEN3_30B_A3B_MOE
    E, K, H, I = cfg["experts"], cfg["top_k"], cfg["hidden"], cfg["inter"]
    mk = lambda t, sh: B.qm_repack(B.qm_quantise(inputs.weights_dev(inputs.seed_for(4, 0, t), sh), B.Q4_G32),
                                   B.LAYOUT_DEVICE)
    wg, wu, wdn = mk("gate", (E, I, H)), mk("up", (E, I, H)), mk("down", (E, H, I))
    wbytes = 3 * E * workloads.q4_bytes(H, I)
    # Cold-cache timing: inside a model the 340 MB of expert weights are
    # evicted by the other layers before the layer runs again, so each timed
    # call follows a 512 MiB fill (larger than L2 + MALL); HIP events bracket
    # the layer's own launches on the current stream.
    flush = torch.empty(512 * 2**20, dtype=torch.uint8, device="cuda")

    def cold_us(run, reps=9):
        st = torch.cuda.current_stream()
        ts = []
        for i in range(reps + 1):
            flush.fill_(i & 0xFF)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            run(ctypes.c_void_p(st.cuda_stream))
            e1.record(st)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3)
        ts = sorted(ts[1:])
        return ts[len(ts) // 2]

    for m in cfg["m_sweep"]:
        x = inputs.activations_dev(inputs.seed_for(4, m, "x"), (m, H))
        lg = inputs.logits_dev(inputs.seed_for(4, m, "logits"), (m, E))
        r = B.qmoe_route(lg, K)
        yv = torch.empty((m, H), device="cuda")
        ws = torch.empty(B.qmoe_workspace_bytes(m, E, K, H, I), dtype=torch.uint8, device="cuda")
        def run(s, x=x, lg=lg, r=r, yv=yv, ws=ws):
            B.qmoe_route(lg, K, out=r, stream=_Raw(s))
            B.qmoe_grouped_gemm(wg, wu, wdn, x, r, out=yv, workspace=ws, stream=_Raw(s))
        g = capture(torch, run)
        t, _ = time_graph(torch, g, max(steps // 2, 5), warmup)
        n = max(steps // 2, 5)
        flops = 2.0 * m * K * 3 * H * I
        tf = flops * n / t / 1e12
        ai = flops / wbytes
        attainable = min(MFMA_F16_PEAK_TFLOPS, ai * HBM_PEAK_GBS / 1e3)
        out[f"qwen3-30b-a3b_moe_m{m}"] = {"tokens_per_s": round(m * n / t, 1), "layer_us": round(t / n * 1e6, 2),
                                          "TFLOPs": round(tf, 2), "frac_mfma_peak": round(tf / MFMA_F16_PEAK_TFLOPS, 4),
                                          "frac_attainable": round(tf / attainable, 4),
                                          "weight_GBps": round(wbytes * n / t / 1e9, 1)}
        tc = cold_us(run)
        out[f"qwen3-30b-a3b_moe_m{m}"].update({"layer_us_cold_cache": round(tc, 2),
                                               "weight_GBps_cold_cache": round(wbytes / tc / 1e3, 1)})
        log(f"moe m={m}: {out[f'qwen3-30b-a3b_moe_m{m}']}")
        del g
    del flush
    # The same layer at M = 512 with the experts in the other quantised
    # formats (graph replay; weight bytes = codes + one fp16 scale per 32).
    del wg, wu, wdn
    m = 512
    x = inputs.activations_dev(inputs.seed_for(4, m, "x"), (m, H))
    lg = inputs.logits_dev(inputs.seed_for(4, m, "logits"), (m, E))
    r = B.qmoe_route(lg, K)
    yv = torch.empty((m, H), device="cuda")
    ws = torch.empty(B.qmoe_workspace_bytes(m, E, K, H, I), dtype=torch.uint8, device="cuda")
    by_fmt = {}
    for name, fmt, bits in (("q2", B.Q2_G32, 2), ("q3", B.Q3_G32, 3), ("q4", B.Q4_G32, 4), ("q5", B.Q5_G32, 5),
                            ("q6", B.Q6_G32, 6), ("q8", B.Q8_G32, 8)):
        mkf = lambda t, sh: B.qm_repack(B.qm_quantise(inputs.weights_dev(inputs.seed_for(4, 0, t), sh), fmt),
                                        B.LAYOUT_DEVICE)
        fg, fu, fd = mkf("gate", (E, I, H)), mkf("up", (E, I, H)), mkf("down", (E, H, I))
        def run(s, fg=fg, fu=fu, fd=fd):
            B.qmoe_route(lg, K, out=r, stream=_Raw(s))
            B.qmoe_grouped_gemm(fg, fu, fd, x, r, out=yv, workspace=ws, stream=_Raw(s))
        g = capture(torch, run)
        n = max(steps // 2, 5)
        t, _ = time_graph(torch, g, n, warmup)
        fbytes = 3 * E * H * I * (bits + 0.5) / 8
        tf = 2.0 * m * K * 3 * H * I * n / t / 1e12
        by_fmt[name] = {"layer_us": round(t / n * 1e6, 2), "TFLOPs": round(tf, 1),
                        "frac_mfma_peak": round(tf / MFMA_F16_PEAK_TFLOPS, 4),
                        "weight_MB": round(fbytes / 1e6, 1), "weight_GBps": round(fbytes * n / t / 1e9, 1)}
        del g, fg, fu, fd
    out["qwen3-30b-a3b_moe_m512_by_format"] = by_fmt
    log(f"moe m=512 by format: {by_fmt}")
    return out


class _Raw:
    """Adapter so binding functions accept a raw stream pointer."""

    def __init__(self, ptr):
        self.cuda_stream = ptr.value


# ------------------------------------------------------ HBM traffic

TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gemv_q4_llama3.2-3b_decode_pmc.txt")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2607_00501_amd", "csrc", f) for f in ("gemv.hip", "qm_internal.h")]


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_from_profile(kernel):
    """Mean HBM bytes per launch of `kernel` from the committed rocprofv3
    counter summary (FETCH_SIZE + WRITE_SIZE, each scaled by the copy-kernel
    factor), or None if the GEMV source changed since the counters were
    taken or the summary has no line for this kernel."""
    try:
        with open(TRAFFIC_PROFILE) as f:
            for line in f:
                if not line.startswith("traffic:"):
                    continue
                fields = dict(kv.split("=", 1) for kv in line.rstrip("\n").split("\t")[1:])
                if fields.get("kernel") == kernel and fields.get("kernel_source_sha256") == kernel_source_hash():
                    return int(float(fields["hbm_bytes_per_launch"]))
    except (OSError, KeyError, ValueError):
        pass
    return None


def calibration(torch):
    """Achievable rates on this part, measured with torch's own kernels (not
    this library): a streaming copy of 1 GiB (read + write bytes over the
    time, the best of five passes) and an fp16 matmul 8192 x 8192 x 8192
    (hipBLASLt).  Context for the roofline fractions, which stay against the
    spec peaks."""
    st = torch.cuda.current_stream()

    def best_ms(fn, reps):
        fn()
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            fn()
            e1.record(st)
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1))
        return best
    a = torch.ones(256 * 2**20, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    copy_ms = best_ms(lambda: b.copy_(a), 5)
    copy_gbs = 2 * a.numel() * 4 / copy_ms / 1e6
    del a, b
    n = 8192
    x = torch.randn((n, n), device="cuda").half()
    w = torch.randn((n, n), device="cuda").half()
    mm_ms = best_ms(lambda: torch.matmul(x, w), 5)
    mm_tf = 2 * n ** 3 / mm_ms / 1e9
    del x, w
    torch.cuda.empty_cache()
    return {"stream_copy_GBps": round(copy_gbs, 1), "f16_matmul_TFLOPs": round(mm_tf, 1),
            "how": "torch on this GPU: copy of 1 GiB (read + write bytes), fp16 matmul 8192^3 (hipBLASLt); best of 5"}


# ---------------------------------------------------------------- main

def gemv_kernel_names(B):
    """K->N -> the Q4 GEMV kernel the library launches for that shape (its
    own per-chip plan, as reported by qm_device_config)."""
    import re
    return {m.group(1): m.group(2) for m in re.finditer(r"gemv_q4\((\d+->\d+)\)=(\S[^<]*<[^>]*>)",
                                                         B.qm_device_config())}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--extra", choices=["all", "none", "tg", "decode", "prefill", "moe", "qwen-stack"], default="all",
                    help="other workloads to time after the headline step (subsets for profiling)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the quantised matmul path "
                                   "has no multi-GPU component; run with --gpus 1"}))
        sys.exit(2)

    import torch
    from paper_2607_00501_amd import binding as B
    from paper_2607_00501_amd import inputs, workloads

    B.lib()                                   # raises if the HIP library is missing
    torch.cuda.set_device(0)
    log(f"device config: {B.qm_device_config()}")
    names = gemv_kernel_names(B)

    # copy kernel of known size, for scaling the HBM byte counters
    a = torch.empty(64 << 20, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    torch.neg(a, out=b)
    torch.cuda.synchronize()
    del a, b

    model = workloads.LLAMA32_3B
    calls, nbytes = build_decode_stack(model, 2, B.Q4_G32, torch, B, inputs, workloads)
    log(f"llama-3.2-3b stack ready: {len(calls)} GEMVs, {nbytes} weight bytes")
    g = capture(torch, lambda s: [c(s) for c in calls])
    secs, wall = time_graph(torch, g, args.steps, args.warmup)
    gbs = nbytes * args.steps / secs / 1e9
    log(f"step: {secs / args.steps * 1e3:.4f} ms, {gbs:.1f} GB/s (wall {wall:.3f} s)")
    # spread over single replays (event pair around each)
    st = torch.cuda.current_stream()
    per = []
    for _ in range(min(args.steps, 50)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        g.replay()
        e1.record(st)
        torch.cuda.synchronize()
        per.append(e0.elapsed_time(e1))
    per.sort()
    pct = lambda q: per[min(len(per) - 1, int(q * len(per)))]
    del g

    # Per projection shape: all launches of that shape in the step, back to
    # back in one graph (stack order, each with its own weights), HIP events
    # on the launch stream -> mean launch duration.  The dominant kernel is
    # the shape with the largest share of the step (launches x duration).
    shapes = {}
    for c, (layer, name, k, n) in zip(calls, workloads.stack_calls(model)):
        shapes.setdefault((k, n), []).append(c)
    per_shape = {}
    for (k, n), cs in shapes.items():
        gs = capture(torch, lambda s, cs=cs: [c(s) for c in cs])
        reps = max(3, 200 // len(cs))
        t, _ = time_graph(torch, gs, reps, 2)
        us = t / reps / len(cs) * 1e6
        bpl = workloads.q4_bytes(k, n)
        per_shape[f"{k}->{n}"] = {"kernel": names.get(f"{k}->{n}", "?"), "launches_per_step": len(cs),
                                  "mean_launch_us": round(us, 3), "algorithmic_bytes_per_launch": bpl,
                                  "GBps": round(bpl / us / 1e3, 1), "frac_hbm_peak": round(bpl / us / 1e3 / HBM_PEAK_GBS, 4),
                                  "us_per_step": round(us * len(cs), 2)}
        del gs
    dom_shape = max(per_shape, key=lambda kk: per_shape[kk]["us_per_step"])
    dom = per_shape[dom_shape]
    achieved = dom["algorithmic_bytes_per_launch"] / (dom["mean_launch_us"] * 1e-6) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic_from_profile(dom["kernel"]),
                "kernel": f"{dom['kernel']} (Q4 GEMV {dom_shape}, {dom['launches_per_step']} launches per step)",
                "mean_launch_us": dom["mean_launch_us"],
                "algorithmic_bytes_per_launch": dom["algorithmic_bytes_per_launch"],
                "timing": "HIP events over a graph of all launches of this shape in the step, back to back",
                "per_shape": per_shape}
    # The lm_head back to back over 3 copies (665 MB per cycle, beyond the MALL).
    lm_bytes = workloads.q4_bytes(*model["lm_head"])
    lm_us = steady_launch_us(torch, B, calls[-1], copies=3, reps=12)
    roofline.update({"lm_head_steady_us": round(lm_us, 3),
                     "lm_head_steady_GBps": round(lm_bytes / lm_us / 1e3, 1),
                     "lm_head_steady_frac": round(lm_bytes / lm_us / 1e3 / HBM_PEAK_GBS, 4)})
    cal = calibration(torch)
    roofline["frac_of_measured_stream_copy"] = round(achieved / cal["stream_copy_GBps"], 4)
    log(f"roofline: {roofline}")
    log(f"calibration: {cal}")

    extra = {}
    if args.extra != "none":
        del calls
        torch.cuda.empty_cache()
        extra = extra_workloads(torch, B, inputs, workloads, args.steps, args.warmup, args.extra)

    cpu = cpu_baseline(args.cpu_seconds)
    log(f"cpu baseline: {cpu}")

    line = {
        "metric": "Q4 decode GEMV weight GB/s (% of HBM peak); prefill/MoE GEMM TFLOP/s",
        "value": round(gbs, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(secs / args.steps * 1e3, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f16",
        "data": "synthetic (seeded N(0,0.02^2) weights quantised on the GPU, N(0,1) fp16 activations)",
        "config": {"workload": "llama-3.2-3b decode stack, batch 1, Q4 group-32: 28 layers x 7 GEMVs + "
                               "lm_head 3072->128256 (197 GEMV calls per token)",
                   "weight_bytes_per_step": nbytes, "tokens_per_s": round(args.steps / secs, 2),
                   "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
                   "ms_per_step_p10_p50_p90": [round(pct(0.1), 4), round(pct(0.5), 4), round(pct(0.9), 4)],
                   "timing": "hip graph replay, HIP events",
                   "arithmetic": "Q4 codes dequantised to fp16 in registers, fp16 products, fp32 accumulation"},
        "roofline": roofline,
        "calibration": cal,
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
