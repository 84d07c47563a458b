"""Seeded synthetic inputs shared by the oracle side and the GPU side.

This module holds no arithmetic of the decoding method. It only draws numbers:
model weights shaped like the paper's backbones (Dream-7B / Qwen2.5-7B layout,
LLaDA-8B layout, and a tiny 2-layer decoder), and uniform-random prompt tokens.
The paper's evaluation prompts (GSM8K, MATH, HumanEval, MBPP) and its trained
D2F weights are not available; these random stand-ins keep their shapes only.

Generator (counter-based, so CPU and GPU draw bit-identical values):
  * SplitMix64 (Steele, Lea, Flood 2014; Vigna's reference splitmix64.c):
    state_i = key + (i + 1) * 0x9E3779B97F4A7C15 (mod 2^64), then the
    published three-step xor-shift-multiply finaliser.
  * key = splitmix64_first(seed * 2^32 + stream_id): one stream per tensor.
  * weight: Irwin-Hall(4) over the four 16-bit fields of the 64-bit output,
    w = sigma * sqrt(3) * (sum - 131070) / 65536 (mean 0, std sigma, bounded at
    +-3.46 sigma), evaluated as int64 -> float64 multiply -> float32 (RNE).
  * token: ((z >> 32) * (V - 1)) >> 32, uniform on [0, V - 2] (mask id V - 1
    excluded).

All arithmetic is int64 with two's-complement wrap plus one IEEE float64
multiply, so torch on CPU and on the GPU give the same bits.
"""
from __future__ import annotations

import math

import torch

GOLDEN = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB
M64 = (1 << 64) - 1

# ---------------------------------------------------------------- configs
from .shapes import CONFIGS, config  # noqa: E402,F401


# ------------------------------------------------------------- generator
def _i64(c: int) -> int:
    c &= M64
    return c - (1 << 64) if c >= (1 << 63) else c


def splitmix64_scalar(state: int) -> tuple[int, int]:
    """One step of the reference generator on Python ints: (new_state, output)."""
    state = (state + GOLDEN) & M64
    z = state
    z = ((z ^ (z >> 30)) * MIX1) & M64
    z = ((z ^ (z >> 27)) * MIX2) & M64
    return state, z ^ (z >> 31)


def _lshr(z: torch.Tensor, s: int) -> torch.Tensor:
    return torch.bitwise_right_shift(z, s) & ((1 << (64 - s)) - 1)


def _mix(z: torch.Tensor) -> torch.Tensor:
    z = (z ^ _lshr(z, 30)) * _i64(MIX1)
    z = (z ^ _lshr(z, 27)) * _i64(MIX2)
    return z ^ _lshr(z, 31)


def stream_key(seed: int, stream_id: int) -> int:
    return splitmix64_scalar(((seed & 0xFFFFFFFF) << 32) | (stream_id & 0xFFFFFFFF))[1]


def raw64(key: int, start: int, n: int, device="cpu") -> torch.Tensor:
    """Outputs start..start+n-1 of the SplitMix64 sequence seeded with `key` (int64 bits)."""
    i = torch.arange(start + 1, start + n + 1, dtype=torch.int64, device=device)
    return _mix(i * _i64(GOLDEN) + _i64(key))


_CHUNK = 1 << 24


def irwin_hall(key: int, n: int, std: float, device="cpu") -> torch.Tensor:
    """n float32 draws with mean 0 and standard deviation `std`."""
    out = torch.empty(n, dtype=torch.float32, device=device)
    scale = std * math.sqrt(3.0) / 65536.0
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        z = raw64(key, s, e - s, device)
        tot = (z & 0xFFFF) + (_lshr(z, 16) & 0xFFFF) + (_lshr(z, 32) & 0xFFFF) + _lshr(z, 48)
        out[s:e] = ((tot - 131070).to(torch.float64) * scale).to(torch.float32)
    return out


def uniform_tokens(key: int, n: int, vocab: int, device="cpu") -> torch.Tensor:
    """n int64 tokens uniform on [0, vocab - 2]."""
    z = raw64(key, 0, n, device)
    return (_lshr(z, 32) * (vocab - 1)) >> 32


# ------------------------------------------------------------- tensors
_STREAM = {"wq": 1, "wk": 2, "wv": 3, "bq": 4, "bk": 5, "bv": 6, "wo": 7,
           "w_gate": 8, "w_up": 9, "w_down": 10}
_EMBED, _LM_HEAD, _PROMPT = 60001, 60002, 60003


def _draw(seed, sid, shape, std, device, dtype):
    n = 1
    for s in shape:
        n *= s
    t = irwin_hall(stream_key(seed, sid), n, std, device).reshape(shape)
    return t if dtype == torch.float32 else t.to(dtype)


def layer_weights(cfg: dict, layer: int, seed: int = 0, device="cpu", dtype=torch.float32) -> dict:
    """One decoder layer in PyTorch [out, in] layout."""
    H, Hq, Hkv, d, F = cfg["hidden"], cfg["heads"], cfg["kv_heads"], cfg["head_dim"], cfg["ffn"]
    std = cfg["std"]
    shapes = {"wq": (Hq * d, H), "wk": (Hkv * d, H), "wv": (Hkv * d, H), "wo": (H, Hq * d),
              "w_gate": (F, H), "w_up": (F, H), "w_down": (H, F)}
    if cfg["qkv_bias"]:
        shapes.update({"bq": (Hq * d,), "bk": (Hkv * d,), "bv": (Hkv * d,)})
    out = {k: _draw(seed, 64 * (layer + 1) + _STREAM[k], s, std, device, dtype) for k, s in shapes.items()}
    out["ln1"] = torch.ones(H, dtype=dtype, device=device)
    out["ln2"] = torch.ones(H, dtype=dtype, device=device)
    return out


def embed_weight(cfg, seed=0, device="cpu", dtype=torch.float32):
    return _draw(seed, _EMBED, (cfg["vocab"], cfg["hidden"]), cfg["std"], device, dtype)


def lm_head_weight(cfg, seed=0, device="cpu", dtype=torch.float32):
    return _draw(seed, _LM_HEAD, (cfg["vocab"], cfg["hidden"]), cfg["lm_std"], device, dtype)


def model_weights(cfg: dict, seed: int = 0, device="cpu", dtype=torch.float32) -> dict:
    """All weights: {'embed', 'layers': [...], 'final_norm', 'lm_head'}."""
    return {
        "embed": embed_weight(cfg, seed, device, dtype),
        "layers": [layer_weights(cfg, l, seed, device, dtype) for l in range(cfg["layers"])],
        "final_norm": torch.ones(cfg["hidden"], dtype=dtype, device=device),
        "lm_head": lm_head_weight(cfg, seed, device, dtype),
    }


def prompt(cfg: dict, n: int, seed: int = 1, device="cpu") -> torch.Tensor:
    return uniform_tokens(stream_key(seed, _PROMPT), n, cfg["vocab"], device)


def to_bf16_values(w):
    """Round every tensor of a weight dict to bf16 (RNE) and back to float32."""
    if isinstance(w, dict):
        return {k: to_bf16_values(v) for k, v in w.items()}
    if isinstance(w, list):
        return [to_bf16_values(v) for v in w]
    return w.to(torch.bfloat16).to(torch.float32)
