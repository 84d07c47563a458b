"""Model shapes of the synthetic workloads (no PyTorch, so that torch-free
harnesses can read them by file path)."""
from __future__ import annotations

import math

# ---------------------------------------------------------------- configs
# Shapes follow the public configs of the paper's backbones (the paper names
# the models only). mask_id = V - 1 for every config.
CONFIGS = {
    # 2 layers, hidden 256, 4 q / 2 kv heads, head_dim 64, FFN 704, vocab 1024.
    "tiny": dict(layers=2, hidden=256, heads=4, kv_heads=2, head_dim=64, ffn=704,
                 vocab=1024, rms_eps=1e-6, rope_theta=1e4, qkv_bias=True,
                 std=0.02, lm_std=0.5),
    # Several GEMM tiles, ragged vocab (not a multiple of 128), GQA 4:1. The
    # LM head is spread to a logit std of 4 (lm_std 4 / sqrt(hidden)) so that
    # confidences are informative (conf > 0.9 occurs) while bf16 rounding
    # noise, which grows with the spread, stays inside the 2e-2 confidence
    # tolerance over multi-iteration trajectories as well.
    "small": dict(layers=3, hidden=512, heads=8, kv_heads=2, head_dim=64, ffn=1408,
                  vocab=3000, rms_eps=1e-6, rope_theta=1e4, qkv_bias=True,
                  std=0.02, lm_std=4.0 / math.sqrt(512)),
    # head_dim 128 path with a 2:1 GQA ratio, no biases.
    "small128": dict(layers=2, hidden=512, heads=4, kv_heads=2, head_dim=128, ffn=1024,
                     vocab=2048, rms_eps=1e-5, rope_theta=5e5, qkv_bias=False,
                     std=0.02, lm_std=5.0 / math.sqrt(512)),
    # One-layer models of other widths: rows of 1536 and 6144 values (the
    # RMSNorm kernels' 512-thread and 1024-thread x 2-group row forms), GQA 3:1
    # and 6:1, FFN widths not a multiple of the GEMM tiles' 160 columns.
    "wide1536": dict(layers=1, hidden=1536, heads=12, kv_heads=4, head_dim=128, ffn=4096,
                     vocab=2048, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True,
                     std=0.02, lm_std=4.0 / math.sqrt(1536)),
    "wide6144": dict(layers=1, hidden=6144, heads=48, kv_heads=8, head_dim=128, ffn=8192,
                     vocab=2048, rms_eps=1e-5, rope_theta=5e5, qkv_bias=False,
                     std=0.02, lm_std=4.0 / math.sqrt(6144)),
    # Dream-7B (Qwen2.5-7B layout).
    "dream7b": dict(layers=28, hidden=3584, heads=28, kv_heads=4, head_dim=128, ffn=18944,
                    vocab=152064, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True,
                    std=0.02, lm_std=0.02),
    # Same shape, LM head spread (logit std 5) so that confidences are not all ~1/V.
    "dream7b_spread": dict(layers=28, hidden=3584, heads=28, kv_heads=4, head_dim=128,
                           ffn=18944, vocab=152064, rms_eps=1e-6, rope_theta=1e6,
                           qkv_bias=True, std=0.02, lm_std=5.0 / math.sqrt(3584)),
    # LLaDA-8B layout: MHA, no biases.
    "llada8b": dict(layers=32, hidden=4096, heads=32, kv_heads=32, head_dim=128, ffn=12288,
                    vocab=126464, rms_eps=1e-5, rope_theta=5e5, qkv_bias=False,
                    std=0.02, lm_std=0.02),
    # Same shape, LM head spread (logit std 5, parity cases).
    "llada8b_spread": dict(layers=32, hidden=4096, heads=32, kv_heads=32, head_dim=128,
                           ffn=12288, vocab=126464, rms_eps=1e-5, rope_theta=5e5,
                           qkv_bias=False, std=0.02, lm_std=5.0 / math.sqrt(4096)),
}


def config(name: str, **over) -> dict:
    c = dict(CONFIGS[name])
    c.update(over)
    c["name"] = name
    c["mask_id"] = c["vocab"] - 1
    return c
