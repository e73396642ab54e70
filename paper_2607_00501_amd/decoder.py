"""Host sequencing of one decode step of a dense grouped-query-attention
decoder (the Llama 3.2 / Qwen3 layer) over the library's entry points
(BaseRT Sec. 3.2: a token is embedding, per layer norm -> q/k/v projections
-> RoPE and cache append -> attention -> output projection -> residual and
norm -> SwiGLU feed-forward, then the final norm, the LM head and sampling).

Every arithmetic step runs in the library's kernels; this module owns the
device buffers and issues the calls in order on one stream, with no host
synchronisation, so a step (or several) can be captured in a HIP graph and
the sampled token stays on the device for the next step's embedding.
"""

import math
from dataclasses import dataclass
from typing import List, Optional

import torch

from . import binding as B


@dataclass
class DecoderConfig:
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    inter: int
    vocab: int
    layers: int
    eps: float = 1e-6
    theta: float = 1e6
    # (factor, low_freq_factor, high_freq_factor, original_len): the Llama 3
    # long-context RoPE frequencies (None: plain theta^(-2i/D))
    rope_scaling: Optional[tuple] = None


@dataclass
class LayerWeights:
    wq: B.QWeight
    wk: B.QWeight
    wv: B.QWeight
    wo: B.QWeight
    wg: B.QWeight
    wu: B.QWeight
    wd: B.QWeight
    attn_norm: torch.Tensor   # fp16 [hidden]
    ffn_norm: torch.Tensor    # fp16 [hidden]
    q_norm: Optional[torch.Tensor] = None   # fp16 [head_dim]: per-head q/k RMSNorm (the Qwen3 layer)
    k_norm: Optional[torch.Tensor] = None


class DenseDecoder:
    """Buffers and call order of one decode step.  Weights: device-layout
    quantised projections, fp16 embedding table and norm weights.

    fused: the two RMSNorms of a layer run inside the GEMVs that read them
    (qmatmul_gemv_grouped_rmsnorm, qmatmul_gemv_swiglu_rmsnorm_f16; any
    weight format, hidden <= 4096), with the residual stream alternating between
    two buffers; otherwise each norm is a launch of its own.

    rope_rows_interleaved: W_q and W_k were quantised from rows in
    binding.rope_interleave_rows order; then (with fused) RoPE and the cache
    append run as the epilogue of the q/k/v GEMV
    (qmatmul_gemv_qkv_rmsnorm_rope): 5 launches per layer."""

    def __init__(self, cfg: DecoderConfig, emb: torch.Tensor, layers: List[LayerWeights], norm: torch.Tensor,
                 lm_head: B.QWeight, max_len: int, fused: bool = True, rope_rows_interleaved: bool = False,
                 max_chunk: int = 512):
        self.cfg, self.emb, self.layers, self.norm, self.lm_head = cfg, emb, layers, norm, lm_head
        self.max_len = max_len
        self.max_chunk = max_chunk          # rows of a prompt chunk (prefill)
        self._chunk = None
        dev = emb.device
        f32 = dict(dtype=torch.float32, device=dev)
        f16 = dict(dtype=torch.float16, device=dev)
        c = cfg
        qd, kvd = c.n_q_heads * c.head_dim, c.n_kv_heads * c.head_dim
        self.fused = fused and c.hidden <= 4096
        self.x = torch.zeros(c.hidden, **f32)             # residual stream
        self.x2 = torch.zeros(c.hidden, **f32)            # its other buffer (fused norms)
        self.rope_epi = rope_rows_interleaved
        assert not self.rope_epi or self.fused, "the RoPE epilogue runs in the fused q/k/v GEMV"
        assert not (self.rope_epi and any(ly.q_norm is not None for ly in layers)), \
            "per-head q/k norms need whole heads: use the RoPE kernel (rows not interleaved)"
        # (cos, sin) of every cache position, built once: read by the q/k/v
        # GEMV's RoPE epilogue and by the prompt path's RoPE kernel.
        # every RoPE of the step and of the prompt path reads this table
        self.rope_tab = (B.qdec_rope_table(max_len, c.head_dim, c.theta, device=dev) if c.rope_scaling is None else
                         B.qdec_rope_table_llama3(max_len, c.head_dim, c.theta, c.rope_scaling, device=dev))
        self.h = torch.zeros(c.hidden, **f16)             # normed input of a projection
        self.q, self.k, self.v = torch.zeros(qd, **f32), torch.zeros(kvd, **f32), torch.zeros(kvd, **f32)
        self.q16 = torch.zeros((c.n_q_heads, c.head_dim), **f16)
        self.attn16 = torch.zeros((c.n_q_heads, c.head_dim), **f16)
        self.y_attn = torch.zeros(c.hidden, **f32)
        self.g16 = torch.zeros(c.inter, **f16)
        self.y_ffn = torch.zeros(c.hidden, **f32)
        self.logits = torch.zeros(c.vocab, **f32)
        self.token = torch.zeros(1, dtype=torch.int32, device=dev)
        self.k_cache = torch.zeros((c.layers, c.n_kv_heads, max_len, c.head_dim), **f16)
        self.v_cache = torch.zeros((c.layers, c.n_kv_heads, max_len, c.head_dim), **f16)
        self.ws = torch.empty(B.qattn_decode_workspace_bytes(c.n_q_heads, c.head_dim), dtype=torch.uint8,
                              device=dev)
        self.argmax_ws = torch.empty(B.ARGMAX_WORKSPACE_BYTES, dtype=torch.uint8, device=dev)
        self.scale = 1.0 / math.sqrt(c.head_dim)

    def step(self, pos: int, stream=None) -> None:
        """Consumes self.token (the token at position pos), writes row pos of
        every layer's caches, self.logits, and the greedy next token into
        self.token."""
        c, s = self.cfg, stream
        B.qdec_embed(self.emb, self.token, out=self.x, stream=s)
        if self.fused:
            for li, ly in enumerate(self.layers):
                res = self.y_ffn if li else None
                if self.rope_epi:
                    # x2 = x + y_ffn; q, k, v = W . norm(x2), rotated, k and v into the caches
                    B.qmatmul_gemv_qkv_rmsnorm_rope([ly.wq, ly.wk, ly.wv], self.x, ly.attn_norm, c.eps, self.x2, pos,
                                                    self.rope_tab, self.q16, self.k_cache[li], self.v_cache[li],
                                                    residual=res, stream=s)
                else:
                    # x2 = x + y_ffn; q, k, v = W . norm(x2)
                    B.qmatmul_gemv_grouped_rmsnorm([ly.wq, ly.wk, ly.wv], self.x, ly.attn_norm, c.eps, self.x2,
                                                   residual=res, outs=[self.q, self.k, self.v], stream=s)
                    # RoPE (with the Qwen3 per-head norms) + cache append, then attention
                    B.qdec_rope_append(self.q, self.k, self.v, pos, c.theta, self.k_cache[li], self.v_cache[li],
                                       q_out=self.q16, q_norm=ly.q_norm, k_norm=ly.k_norm, eps=c.eps,
                                       table=self.rope_tab, stream=s)
                B.qattn_decode(self.q16, self.k_cache[li], self.v_cache[li], pos + 1, self.scale, out=self.attn16,
                               workspace=self.ws, stream=s)
                B.qmatmul_gemv(ly.wo, self.attn16.view(-1), out=self.y_attn, stream=s)
                # x = x2 + y_attn; g = swiglu(norm(x))
                B.qmatmul_gemv_swiglu_rmsnorm_f16(ly.wg, ly.wu, self.x2, ly.ffn_norm, c.eps, self.x,
                                                  residual=self.y_attn, out=self.g16, stream=s)
                B.qmatmul_gemv(ly.wd, self.g16, out=self.y_ffn, stream=s)
            self._head(s)
            return
        for li, ly in enumerate(self.layers):
            B.qdec_rmsnorm(self.x, ly.attn_norm, c.eps, residual=self.y_ffn if li else None, out=self.h, stream=s)
            B.qmatmul_gemv_grouped([ly.wq, ly.wk, ly.wv], [self.h] * 3, [self.q, self.k, self.v], stream=s)
            B.qdec_rope_append(self.q, self.k, self.v, pos, c.theta, self.k_cache[li], self.v_cache[li],
                               q_out=self.q16, q_norm=ly.q_norm, k_norm=ly.k_norm, eps=c.eps,
                               table=self.rope_tab, stream=s)
            B.qattn_decode(self.q16, self.k_cache[li], self.v_cache[li], pos + 1, self.scale, out=self.attn16,
                           workspace=self.ws, stream=s)
            B.qmatmul_gemv(ly.wo, self.attn16.view(-1), out=self.y_attn, stream=s)
            B.qdec_rmsnorm(self.x, ly.ffn_norm, c.eps, residual=self.y_attn, out=self.h, stream=s)
            B.qmatmul_gemv_swiglu(ly.wg, ly.wu, self.h, out=self.g16, stream=s)
            B.qmatmul_gemv(ly.wd, self.g16, out=self.y_ffn, stream=s)
        self._head(s)

    def _head(self, s) -> None:
        B.qdec_rmsnorm(self.x, self.norm, self.cfg.eps, residual=self.y_ffn, out=self.h, stream=s)
        B.qmatmul_gemv(self.lm_head, self.h, out=self.logits, stream=s)
        B.qdec_argmax(self.logits, out=self.token, workspace=self.argmax_ws, stream=s)

    def _chunk_buffers(self, m: int) -> dict:
        """Views of the prompt-chunk buffers for m rows.  The buffers hold
        max_chunk rows and are allocated on the first prefill only (a decoder
        that never prefills pays nothing), so later chunks allocate nothing
        (Sec. 3.2: no allocation in the loop; Sec. 3.4: bounded chunks)."""
        c = self.cfg
        qd, kvd = c.n_q_heads * c.head_dim, c.n_kv_heads * c.head_dim
        shapes = dict(x=((c.hidden,), torch.float32), h=((c.hidden,), torch.float16),
                      q=((qd,), torch.float32), k=((kvd,), torch.float32), v=((kvd,), torch.float32),
                      qh=((qd,), torch.float16), o16=((qd,), torch.float16),
                      ya=((c.hidden,), torch.float32), g=((c.inter,), torch.float32),
                      u=((c.inter,), torch.float32), sw=((c.inter,), torch.float16), y=((c.hidden,), torch.float32))
        if self._chunk is None:
            dev = self.emb.device
            self._chunk = {n: torch.empty(self.max_chunk * sh[0], dtype=dt, device=dev)
                           for n, (sh, dt) in shapes.items()}
            # Key-split partials of the prefill attention, sized for a full
            # chunk at position 0 (the deepest causal triangle); other chunks
            # split within it.
            nb = B.qattn_prefill_workspace_bytes(c.n_q_heads, c.head_dim, self.max_chunk, 0)
            self._chunk["attn_ws"] = torch.empty(max(nb, 16), dtype=torch.uint8, device=dev)
        b = self._chunk
        rows = lambda n: b[n][:m * shapes[n][0][0]].view(m, shapes[n][0][0])
        heads = lambda n: b[n][:m * qd].view(c.n_q_heads, m, c.head_dim)
        out = {n: rows(n) for n in shapes if n != "qh"}
        out.update(qh=heads("qh"), attn_ws=b["attn_ws"])
        return out

    def prefill(self, tokens: torch.Tensor, p0: int = 0, stream=None) -> None:
        """A prompt chunk (Sec. 3.4): tokens (int32 [m], device, 1 <= m <=
        max_chunk) at positions p0 .. p0 + m - 1 through every layer with the
        prefill GEMMs and causal attention; writes those cache rows, the last
        token's logits and the greedy next token into self.token.  Longer
        prompts go through in several chunks."""
        c, s = self.cfg, stream
        m = tokens.numel()
        if not 1 <= m <= self.max_chunk:
            raise ValueError(f"prefill chunk of {m} tokens: must be 1 .. max_chunk={self.max_chunk}")
        b = self._chunk_buffers(m)
        x = B.qdec_embed_rows(self.emb, tokens, out=b["x"], stream=s)     # fp32 [m][H] residual stream
        y = None
        for li, ly in enumerate(self.layers):
            h = B.qdec_rmsnorm(x, ly.attn_norm, c.eps, residual=y, out=b["h"], stream=s)
            q, k, v = B.qmatmul_gemm_grouped([ly.wq, ly.wk, ly.wv], h, outs=[b["q"], b["k"], b["v"]], stream=s)
            qh = B.qdec_rope_append_rows(q, k, v, p0, c.theta, self.k_cache[li], self.v_cache[li],
                                         interleaved=self.rope_epi, q_out=b["qh"], q_norm=ly.q_norm,
                                         k_norm=ly.k_norm, eps=c.eps, table=self.rope_tab, stream=s)
            o16 = B.qattn_prefill_rows_f16(qh, self.k_cache[li], self.v_cache[li], p0, self.scale, out=b["o16"],
                                           workspace=b["attn_ws"], stream=s)
            ya = B.qmatmul_gemm(ly.wo, o16, out=b["ya"], stream=s)
            h = B.qdec_rmsnorm(x, ly.ffn_norm, c.eps, residual=ya, out=b["h"], stream=s)
            g, u = B.qmatmul_gemm_grouped([ly.wg, ly.wu], h, outs=[b["g"], b["u"]], stream=s)
            y = B.qmatmul_gemm(ly.wd, B.qdec_swiglu_f16(g, u, out=b["sw"], stream=s), out=b["y"], stream=s)
        B.qdec_rmsnorm(x[m - 1], self.norm, c.eps, residual=y[m - 1], out=self.h, stream=s)
        B.qmatmul_gemv(self.lm_head, self.h, out=self.logits, stream=s)
        B.qdec_argmax(self.logits, out=self.token, workspace=self.argmax_ws, stream=s)
