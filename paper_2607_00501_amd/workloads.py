"""Layer shapes of the benchmark workloads (K -> N per projection).

The model shapes are the ones the paper evaluates (Sec. 4.1: Qwen3-0.6B,
Llama-3.2-1B / 3B decode and prefill, Qwen3-30B-A3B MoE prefill); weights
are synthetic.
"""

from __future__ import annotations

# (name, K, N) per projection of one layer
QWEN3_06B_LAYER = [("q", 1024, 2048), ("k", 1024, 1024), ("v", 1024, 1024), ("o", 2048, 1024),
                   ("gate", 1024, 3072), ("up", 1024, 3072), ("down", 3072, 1024)]
QWEN3_06B = dict(name="qwen3-0.6b decode stack", layers=28, layer=QWEN3_06B_LAYER,
                 lm_head=(1024, 151936))

LLAMA32_3B_LAYER = [("q", 3072, 3072), ("k", 3072, 1024), ("v", 3072, 1024), ("o", 3072, 3072),
                    ("gate", 3072, 8192), ("up", 3072, 8192), ("down", 8192, 3072)]
LLAMA32_3B = dict(name="llama-3.2-3b decode stack", layers=28, layer=LLAMA32_3B_LAYER,
                  lm_head=(3072, 128256))

LLAMA32_1B_LAYER = [("q", 2048, 2048), ("k", 2048, 512), ("v", 2048, 512), ("o", 2048, 2048),
                    ("gate", 2048, 8192), ("up", 2048, 8192), ("down", 8192, 2048)]
LLAMA32_1B_PREFILL = dict(name="llama-3.2-1b prefill gemms", layers=16, layer=LLAMA32_1B_LAYER,
                          m_sweep=(128, 512, 2048))

QWEN3_30B_A3B_MOE = dict(name="qwen3-30b-a3b moe layer", hidden=2048, inter=768, experts=128,
                         top_k=8, m_sweep=(128, 512, 2048))

# Whole dense decoders (attention geometry, FFN width, vocabulary) for the
# end-to-end decode benchmark: tg128, 128 greedy tokens from an empty cache
# (Sec. 4.1).  RoPE: each model's theta; the Llama 3.2 models with their
# long-context frequency rule (factor 32, low / high frequency factors 1 / 4,
# original length 8192).
QWEN3_06B_DECODER = dict(name="qwen3-0.6b", hidden=1024, n_q_heads=16, n_kv_heads=8, head_dim=128, inter=3072,
                         vocab=151936, layers=28, theta=1e6)
LLAMA32_1B_DECODER = dict(name="llama-3.2-1b", hidden=2048, n_q_heads=32, n_kv_heads=8, head_dim=64, inter=8192,
                          vocab=128256, layers=16, theta=5e5,
                          rope_scaling=(32, 1, 4, 8192))
LLAMA32_3B_DECODER = dict(name="llama-3.2-3b", hidden=3072, n_q_heads=24, n_kv_heads=8, head_dim=128, inter=8192,
                          vocab=128256, layers=28, theta=5e5,
                          rope_scaling=(32, 1, 4, 8192))

SINGLE_GEMV = dict(name="single q4 gemv 1024x1024", k=1024, n=1024)


def stack_calls(model: dict):
    """Every GEMV of one decode step in issue order: (layer, name, K, N)."""
    calls = [(l, name, k, n) for l in range(model["layers"]) for name, k, n in model["layer"]]
    if model.get("lm_head"):
        k, n = model["lm_head"]
        calls.append((model["layers"], "lm_head", k, n))
    return calls


def q4_bytes(k: int, n: int) -> int:
    """Algorithmic Q4 weight bytes of a K -> N matrix: half a byte per code
    plus a 2-byte scale per 32 codes."""
    return n * (k // 2) + n * (k // 32) * 2


def q8_bytes(k: int, n: int) -> int:
    return n * k + n * (k // 32) * 2


FORMAT_BITS = {1: 4, 2: 8, 3: 2, 4: 3, 5: 5, 6: 6, 7: 16, 8: 16}   # format id -> bits per weight
FORMAT_NAMES = {1: "q4", 2: "q8", 3: "q2", 4: "q3", 5: "q5", 6: "q6", 7: "f16", 8: "bf16"}


def weight_bytes(fmt: int, k: int, n: int) -> int:
    """Algorithmic weight bytes of a K -> N matrix in any format: b/8 bytes
    per code, plus a 2-byte scale per 32 codes for the integer formats."""
    b = FORMAT_BITS[fmt]
    return n * k * b // 8 + (0 if b == 16 else n * (k // 32) * 2)
