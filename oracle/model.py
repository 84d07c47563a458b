"""Oracle dLLM forward for one active block of a batch of branches.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py). Plain numpy, float64.

What it computes (the paper, arXiv 2512.16229):
  * Sec. 3.1: the model p_theta gives a predictive distribution per masked
    position; a candidate x0_hat is drawn from it and Conf(.) scores each
    position. Reading used here (the paper does not define Conf further):
    greedy candidate (argmax token) and Conf = its softmax probability. The
    mask token is excluded from the support, so a filled position never holds
    the mask id.
  * Alg. 1 step 3: all branches of the active block go through one batched
    forward pass.
  * Sec. 3.3: attention inside the active block is full (bidirectional); every
    block row also sees the whole committed prefix; branches never see each
    other (each is its own sequence).
  * Sec. 3.4 (LoPA-Dist-NV): a static, pre-allocated KV cache holds the prefix;
    each branch's block K/V are produced by the forward and the winner's are
    committed to the cache afterwards.

The backbone is a Qwen2.5 / LLaMA-style pre-norm decoder (the paper's models,
Dream-7B and DiffuCoder-7B, use this layout; the paper names only the models):
RMSNorm -> Q/K/V projections (+ optional bias) -> rotate-half RoPE on q and k
-> grouped-query softmax attention -> output projection + residual -> RMSNorm
-> SwiGLU MLP + residual; final RMSNorm -> untied LM head.

Precision modes:
  * "pure": float64 everywhere from the weights as given.
  * "faithful": float64 arithmetic, but values are rounded to bf16 (RNE, via
    float32) where a bf16 implementation stores them: weights, the input of
    every projection (norm outputs, attention output, SwiGLU output), q, k and
    v after bias/RoPE, and the softmax numerators exp(s - rowmax) that multiply
    V (the row max is the global max over the row's keys; the denominator is
    the sum of the unrounded numerators).
  * "fp8_mlp": "faithful", except that the MLP projections run in FP8 (W8A8,
    oracle/fp8.py): gate / up / down weights quantised per output channel, the
    normed input of gate/up quantised per row from its unrounded value, the
    SwiGLU output (stored bf16) quantised per row before the down projection.
  * "fp8": "fp8_mlp", and the QKV projection and the LM head in FP8 as well
    (their weights per output channel, their normed inputs per row from the
    unrounded values); the output projection stays bf16.
"""
from __future__ import annotations

import numpy as np

from .fp8 import fp8_matmul, quantize_rows


def bf16_round(x) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even), via float32; returns float64."""
    x32 = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = x32.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    nan = np.isnan(x32)
    if nan.any():
        out[nan] = np.nan
    return out


def _np(t) -> np.ndarray:
    """torch tensor or array -> float64 numpy array."""
    if hasattr(t, "detach"):
        t = t.detach().to("cpu")
        if str(t.dtype) in ("torch.bfloat16", "torch.float16"):
            t = t.float()
        t = t.numpy()
    return np.asarray(t, dtype=np.float64)


def rms_norm(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * w over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def rope_angles(positions: np.ndarray, d: int, theta: float) -> np.ndarray:
    """angle[p, j] = pos_p * theta^(-2j/d), j < d/2 (rotate-half convention)."""
    inv = theta ** (-np.arange(0, d // 2, dtype=np.float64) * 2.0 / d)
    return np.outer(positions.astype(np.float64), inv)


def apply_rope(x: np.ndarray, ang: np.ndarray) -> np.ndarray:
    """Rotate the pairs (j, j + d/2) of the last axis by ang[..., j].

    x: [..., L, d]; ang: [L, d/2] broadcast over the leading axes."""
    d = x.shape[-1]
    x1, x2 = x[..., : d // 2], x[..., d // 2:]
    c, s = np.cos(ang), np.sin(ang)
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


class KVCache:
    """Static cache: k, v of shape [layers, kv_heads, max_len, head_dim] (float64)."""

    def __init__(self, cfg: dict, max_len: int):
        shp = (cfg["layers"], cfg["kv_heads"], max_len, cfg["head_dim"])
        self.k = np.zeros(shp)
        self.v = np.zeros(shp)
        self.max_len = max_len

    def commit(self, pos: int, k_blk: np.ndarray, v_blk: np.ndarray) -> int:
        """Write one branch's block K/V ([layers, kv_heads, L, d]) at rows [pos, pos+L)."""
        L = k_blk.shape[2]
        if pos + L > self.max_len:
            raise ValueError("cache capacity exceeded")
        self.k[:, :, pos:pos + L] = k_blk
        self.v[:, :, pos:pos + L] = v_blk
        return pos

    def copy(self) -> "KVCache":
        c = KVCache.__new__(KVCache)
        c.k, c.v, c.max_len = self.k.copy(), self.v.copy(), self.max_len
        return c


class OracleModel:
    def __init__(self, cfg: dict, weights: dict, mode: str = "pure"):
        if mode not in ("pure", "faithful", "fp8_mlp", "fp8"):
            raise ValueError(mode)
        self.cfg, self.mode = cfg, mode
        self.fp8_mlp = mode in ("fp8_mlp", "fp8")
        self.fp8_qkv_lm = mode == "fp8"
        r = bf16_round if mode != "pure" else (lambda a: a)
        self.embed = r(_np(weights["embed"]))
        self.lm_head = r(_np(weights["lm_head"]))
        self.final_norm = _np(weights["final_norm"])
        self.layers = []
        for lw in weights["layers"]:
            self.layers.append({k: (r(_np(v)) if k not in ("ln1", "ln2") else _np(v))
                                for k, v in lw.items()})
        quantized = (("w_gate", "w_up", "w_down") if self.fp8_mlp else ()) + \
            (("wq", "wk", "wv") if self.fp8_qkv_lm else ())
        for w in self.layers:
            for key in quantized:
                w[key + "_q"], w[key + "_s"] = quantize_rows(w[key])
        if self.fp8_qkv_lm:
            self.lm_head_q, self.lm_head_s = quantize_rows(self.lm_head)

    def _store(self, a: np.ndarray) -> np.ndarray:
        return bf16_round(a) if self.mode != "pure" else a

    # ------------------------------------------------------------------
    def attention(self, q, k_blk, v_blk, kp, vp, causal_blk: int = 0):
        """Softmax attention of the block rows of each branch.

        q: [nb, Hq, L, d]; k_blk, v_blk: [nb, Hkv, L, d] (the branch's own block);
        kp, vp: [Hkv, P, d] (shared committed prefix). Every row sees all P prefix
        keys and all L keys of its own branch (causal_blk = 0); nothing of other
        branches. causal_blk = c > 0 (the block-wise causal mask of LoPA-Dist's
        Ascend system, Sec. 3.4): the L rows are consecutive sub-blocks of c, and
        a row of sub-block b sees the prefix and the keys of sub-blocks <= b only.
        Returns o: [nb, Hq, L, d]."""
        cfg = self.cfg
        nb, Hq, L, d = q.shape
        group = Hq // cfg["kv_heads"]
        out = np.empty_like(q)
        scale = 1.0 / np.sqrt(d)
        for h in range(Hq):
            g = h // group
            s_pre = np.einsum("bld,pd->blp", q[:, h], kp[g]) * scale           # [nb, L, P]
            s_blk = np.einsum("bld,bmd->blm", q[:, h], k_blk[:, g]) * scale    # [nb, L, L]
            if causal_blk:
                sub = np.arange(L) // causal_blk
                s_blk = np.where(sub[None, :, None] >= sub[None, None, :], s_blk, -np.inf)
            s = np.concatenate([s_pre, s_blk], axis=-1)
            e = np.exp(s - s.max(axis=-1, keepdims=True))
            den = e.sum(axis=-1, keepdims=True)
            num = self._store(e)
            P = kp.shape[1]
            o = (np.einsum("blp,pd->bld", num[..., :P], vp[g])
                 + np.einsum("blm,bmd->bld", num[..., P:], v_blk[:, g]))
            out[:, h] = o / den
        return out

    def forward_block(self, tokens, prefix_len: int, cache: KVCache, keep_hidden: bool = False,
                      n_layers=None, causal_blk: int = 0):
        """One batched forward of nb branches of the active block.

        tokens: int [nb, L] (block rows at positions prefix_len .. prefix_len+L-1).
        Returns dict: conf [nb, L] (float64), pred [nb, L] (int64), k / v
        [nb, layers, Hkv, L, d] (post-RoPE block keys / values), and, if asked,
        'hidden' [nb, L, H] (final-normed rows) and 'logits'. With n_layers set,
        returns only {'x': residual stream after that many layers}. causal_blk:
        the attention mask inside the block (see attention)."""
        cfg = self.cfg
        tokens = np.asarray(tokens, dtype=np.int64)
        nb, L = tokens.shape
        H, Hq, Hkv, d = cfg["hidden"], cfg["heads"], cfg["kv_heads"], cfg["head_dim"]
        P = int(prefix_len)
        ang = rope_angles(np.arange(P, P + L), d, cfg["rope_theta"])
        x = self.embed[tokens]                                          # [nb, L, H]
        ks = np.empty((nb, cfg["layers"], Hkv, L, d))
        vs = np.empty_like(ks)
        for li, w in enumerate(self.layers):
            if n_layers is not None and li == n_layers:
                return {"x": x}
            if self.fp8_qkv_lm:
                h = rms_norm(x, w["ln1"], cfg["rms_eps"])
                q = fp8_matmul(h, w["wq_q"], w["wq_s"])
                k = fp8_matmul(h, w["wk_q"], w["wk_s"])
                v = fp8_matmul(h, w["wv_q"], w["wv_s"])
            else:
                h = self._store(rms_norm(x, w["ln1"], cfg["rms_eps"]))
                q = h @ w["wq"].T
                k = h @ w["wk"].T
                v = h @ w["wv"].T
            if cfg["qkv_bias"]:
                q, k, v = q + w["bq"], k + w["bk"], v + w["bv"]
            q = q.reshape(nb, L, Hq, d).transpose(0, 2, 1, 3)
            k = k.reshape(nb, L, Hkv, d).transpose(0, 2, 1, 3)
            v = v.reshape(nb, L, Hkv, d).transpose(0, 2, 1, 3)
            q = self._store(apply_rope(q, ang))
            k = self._store(apply_rope(k, ang))
            v = self._store(v)
            ks[:, li], vs[:, li] = k, v
            o = self.attention(q, k, v, cache.k[li, :, :P], cache.v[li, :, :P], causal_blk)
            o = self._store(o.transpose(0, 2, 1, 3).reshape(nb, L, Hq * d))
            x = x + o @ w["wo"].T
            if self.fp8_mlp:
                h2 = rms_norm(x, w["ln2"], cfg["rms_eps"])
                a = self._store(silu(fp8_matmul(h2, w["w_gate_q"], w["w_gate_s"]))
                                * fp8_matmul(h2, w["w_up_q"], w["w_up_s"]))
                x = x + fp8_matmul(a, w["w_down_q"], w["w_down_s"])
            else:
                h2 = self._store(rms_norm(x, w["ln2"], cfg["rms_eps"]))
                a = self._store(silu(h2 @ w["w_gate"].T) * (h2 @ w["w_up"].T))
                x = x + a @ w["w_down"].T
        if n_layers is not None:
            return {"x": x}
        if self.fp8_qkv_lm:
            hf = rms_norm(x, self.final_norm, cfg["rms_eps"])
            logits = fp8_matmul(hf, self.lm_head_q, self.lm_head_s)    # [nb, L, V]
        else:
            hf = self._store(rms_norm(x, self.final_norm, cfg["rms_eps"]))
            logits = hf @ self.lm_head.T                                # [nb, L, V]
        conf, pred = confidence(logits, cfg["mask_id"])
        out = {"conf": conf, "pred": pred, "k": ks, "v": vs}
        if keep_hidden:
            out["hidden"], out["logits"] = hf, logits
        return out


def confidence(logits: np.ndarray, mask_id: int):
    """Conf = max softmax probability with the mask token removed from the support;
    pred = its token (lowest id among equal maxima).  Sec. 3.1 (reading: greedy)."""
    lg = np.array(logits, dtype=np.float64, copy=True)
    lg[..., mask_id] = -np.inf
    pred = np.argmax(lg, axis=-1)
    m = np.max(lg, axis=-1)
    conf = 1.0 / np.sum(np.exp(lg - m[..., None]), axis=-1)
    return conf, pred
