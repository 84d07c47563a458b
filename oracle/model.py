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
  * "fp8": "fp8_mlp", and every other projection in FP8 as well: QKV and the
    LM head (their weights per output channel, their normed inputs per row
    from the unrounded values) and the output projection (its weights per
    output channel, the attention output, stored bf16, per row over all heads).
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
    def __init__(self, cfg: dict, weights: dict, mode: str = "pure", keep_layers=True,
                 share=None, bf16_weights: bool = False):
        """weights["layers"] may be any sequence of layer dicts (a lazy one for
        the full-size shapes); each layer is converted on first use and kept
        when keep_layers is True, or the keep_layers most recently used ones
        when it is an int. share: a bf16-mode model built from the same
        bf16-valued weights whose converted layers this one reuses (the same
        float64 values: rounding a bf16 value to bf16 changes nothing).
        bf16_weights: the caller's weights hold bf16 values already, so the
        non-pure modes skip rounding them (the identity on such values)."""
        if mode not in ("pure", "faithful", "fp8_mlp", "fp8"):
            raise ValueError(mode)
        self.cfg, self.mode = cfg, mode
        self.fp8_mlp = mode in ("fp8_mlp", "fp8")
        self.fp8_qkv_lm = mode == "fp8"
        r = bf16_round if (mode != "pure" and not bf16_weights) else (lambda a: a)
        self._r = r
        self.embed = r(_np(weights["embed"]))
        self.lm_head = r(_np(weights["lm_head"]))
        self.final_norm = _np(weights["final_norm"])
        self._raw_layers = weights["layers"]
        self._keep = keep_layers
        self._layers = {}
        if share is not None:
            if self.fp8_mlp or share.fp8_mlp:
                raise ValueError("only bf16-mode models share converted layers")
            self._layers = share._layers
        if self.fp8_qkv_lm:
            self.lm_head_q, self.lm_head_s = quantize_rows(self.lm_head)

    @property
    def layers(self) -> list:
        """All layers, converted (and kept when keep_layers is true)."""
        return [self.layer(i) for i in range(self.cfg["layers"])]

    def layer(self, li: int) -> dict:
        """Layer li's weights as the forward uses them (rounded to bf16 in the
        non-pure modes, plus the E4M3 codes and scales of the quantised ones)."""
        if li in self._layers:
            w = self._layers.pop(li)
            self._layers[li] = w          # most recently used last
            return w
        lw = self._raw_layers[li]
        w = {k: (self._r(_np(v)) if k not in ("ln1", "ln2") else _np(v)) for k, v in lw.items()}
        quantized = (("w_gate", "w_up", "w_down") if self.fp8_mlp else ()) + \
            (("wq", "wk", "wv", "wo") if self.fp8_qkv_lm else ())
        for key in quantized:
            w[key + "_q"], w[key + "_s"] = quantize_rows(w[key])
        if self._keep is True or (self._keep and not isinstance(self._keep, bool)):
            self._layers[li] = w
            if not isinstance(self._keep, bool):
                while len(self._layers) > self._keep:
                    self._layers.pop(next(iter(self._layers)))
        return w

    def _store(self, a: np.ndarray) -> np.ndarray:
        return bf16_round(a) if self.mode != "pure" else a

    # ------------------------------------------------------------------
    def attention(self, q, k_blk, v_blk, kp, vp, causal_blk: int = 0, trace=None):
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
            if trace is not None:
                trace(num)
            P = kp.shape[1]
            o = (np.einsum("blp,pd->bld", num[..., :P], vp[g])
                 + np.einsum("blm,bmd->bld", num[..., P:], v_blk[:, g]))
            out[:, h] = o / den
        return out

    def forward_block(self, tokens, prefix_len: int, cache: KVCache, keep_hidden: bool = False,
                      n_layers=None, causal_blk: int = 0, x_in=None, first_layer: int = 0,
                      trace=None):
        """One batched forward of nb branches of the active block.

        tokens: int [nb, L] (block rows at positions prefix_len .. prefix_len+L-1).
        Returns dict: conf [nb, L] (float64), pred [nb, L] (int64), k / v
        [nb, layers, Hkv, L, d] (post-RoPE block keys / values; layers before
        first_layer are left zero), and, if asked, 'hidden' [nb, L, H]
        (final-normed rows) and 'logits'. With n_layers set, returns only
        {'x': residual stream after that many layers, 'k', 'v'}. causal_blk:
        the attention mask inside the block (see attention).
        x_in / first_layer: start from the given residual stream [nb, L, H]
        before layer first_layer instead of the embeddings (a layer-by-layer
        comparison feeds each layer the other side's input).
        trace: a list that receives (name, layer, value) for every value the
        non-pure modes round to bf16 (the GEMM inputs h, o, h2, a and the
        final hf; q, k, v after bias / RoPE; the softmax numerators p) and for
        the residual stream x after each layer (never rounded)."""
        cfg = self.cfg
        tokens = np.asarray(tokens, dtype=np.int64)
        nb, L = tokens.shape
        H, Hq, Hkv, d = cfg["hidden"], cfg["heads"], cfg["kv_heads"], cfg["head_dim"]
        P = int(prefix_len)
        ang = rope_angles(np.arange(P, P + L), d, cfg["rope_theta"])
        x = self.embed[tokens] if x_in is None else np.array(x_in, dtype=np.float64)  # [nb, L, H]
        ks = np.zeros((nb, cfg["layers"], Hkv, L, d))
        vs = np.zeros_like(ks)
        last = cfg["layers"] if n_layers is None else n_layers
        tr = (lambda name, li, v: trace.append((name, li, v))) if trace is not None else \
            (lambda name, li, v: None)
        for li in range(first_layer, last):
            w = self.layer(li)
            if self.fp8_qkv_lm:
                h = rms_norm(x, w["ln1"], cfg["rms_eps"])
                q = fp8_matmul(h, w["wq_q"], w["wq_s"])
                k = fp8_matmul(h, w["wk_q"], w["wk_s"])
                v = fp8_matmul(h, w["wv_q"], w["wv_s"])
            else:
                h = self._store(rms_norm(x, w["ln1"], cfg["rms_eps"]))
                tr("h", li, h)
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
            tr("q", li, q)
            tr("k", li, k)
            tr("v", li, v)
            ks[:, li], vs[:, li] = k, v
            o = self.attention(q, k, v, cache.k[li, :, :P], cache.v[li, :, :P], causal_blk,
                               trace=(lambda p_, li=li: tr("p", li, p_)))
            o = self._store(o.transpose(0, 2, 1, 3).reshape(nb, L, Hq * d))
            tr("o", li, o)
            if self.fp8_qkv_lm:
                x = x + fp8_matmul(o, w["wo_q"], w["wo_s"])
            else:
                x = x + o @ w["wo"].T
            tr("x1", li, x)
            if self.fp8_mlp:
                h2 = rms_norm(x, w["ln2"], cfg["rms_eps"])
                a = self._store(silu(fp8_matmul(h2, w["w_gate_q"], w["w_gate_s"]))
                                * fp8_matmul(h2, w["w_up_q"], w["w_up_s"]))
                x = x + fp8_matmul(a, w["w_down_q"], w["w_down_s"])
            else:
                h2 = self._store(rms_norm(x, w["ln2"], cfg["rms_eps"]))
                tr("h2", li, h2)
                a = self._store(silu(h2 @ w["w_gate"].T) * (h2 @ w["w_up"].T))
                x = x + a @ w["w_down"].T
            tr("a", li, a)
            tr("x", li, x)
        if n_layers is not None:
            return {"x": x, "k": ks, "v": vs}
        out = self.lm_from_residual(x, trace=trace)
        res = {"conf": out["conf"], "pred": out["pred"], "k": ks, "v": vs}
        if keep_hidden:
            res["hidden"], res["logits"] = out["hidden"], out["logits"]
        return res

    def lm_from_residual(self, x, trace=None) -> dict:
        """Final RMSNorm, LM head and Conf / candidate (Sec. 3.1) of residual
        rows x [..., H]: {'conf', 'pred', 'hidden' (the LM head's input),
        'logits'}."""
        cfg = self.cfg
        x = np.asarray(x, dtype=np.float64)
        if self.fp8_qkv_lm:
            hf = rms_norm(x, self.final_norm, cfg["rms_eps"])
            logits = fp8_matmul(hf, self.lm_head_q, self.lm_head_s)
        else:
            hf = self._store(rms_norm(x, self.final_norm, cfg["rms_eps"]))
            if trace is not None:
                trace.append(("hf", cfg["layers"], hf))
            logits = hf @ self.lm_head.T
        conf, pred = confidence(logits, cfg["mask_id"])
        return {"conf": conf, "pred": pred, "hidden": hf, "logits": logits}


def confidence(logits: np.ndarray, mask_id: int):
    """Conf = max softmax probability with the mask token removed from the support;
    pred = its token (lowest id among equal maxima).  Sec. 3.1 (reading: greedy)."""
    lg = np.array(logits, dtype=np.float64, copy=True)
    lg[..., mask_id] = -np.inf
    pred = np.argmax(lg, axis=-1)
    m = np.max(lg, axis=-1)
    conf = 1.0 / np.sum(np.exp(lg - m[..., None]), axis=-1)
    return conf, pred
