"""A second bf16 implementation of the verify forward for the CPU tests of the
parity tolerances (test infrastructure, not product code).

It rounds to bf16 at exactly the oracle's faithful rounding points (R16), but
does everything between them the way a GPU does: float32 products and sums
(BLAS sgemm), float32 RMSNorm and softmax. It is an independent correct
computation of the same quantity, so its distance from the float64 oracle is
what any correct bf16 implementation must be allowed; the fixed tolerances of
gpu_util are checked against it in test_parity_tolerances.py."""
from __future__ import annotations

import numpy as np

from oracle import OracleModel
from oracle.model import apply_rope, bf16_round, confidence, rope_angles


def mm32(a, b):
    return (a.astype(np.float32) @ b.astype(np.float32)).astype(np.float64)


def norm32(x, w, eps):
    x32 = x.astype(np.float32)
    r = np.float32(1.0) / np.sqrt(np.mean(x32 * x32, -1, keepdims=True, dtype=np.float32)
                                  + np.float32(eps))
    return (x32 * r * w.astype(np.float32)).astype(np.float64)


class Bf16Variant(OracleModel):
    """The oracle's weights (bf16-rounded, mode "faithful"), float32 arithmetic."""

    def __init__(self, cfg, weights):
        super().__init__(cfg, weights, "faithful")

    def attention32(self, q, k_blk, v_blk, kp, vp):
        nb, Hq, L, d = q.shape
        group = Hq // self.cfg["kv_heads"]
        out = np.empty_like(q)
        scale = np.float32(1.0 / np.sqrt(d))
        for h in range(Hq):
            g = h // group
            K = np.concatenate([np.broadcast_to(kp[g], (nb,) + kp[g].shape), k_blk[:, g]], axis=1)
            V = np.concatenate([np.broadcast_to(vp[g], (nb,) + vp[g].shape), v_blk[:, g]], axis=1)
            s = np.einsum("bld,bpd->blp", q[:, h].astype(np.float32), K.astype(np.float32)) * scale
            e = np.exp(s - s.max(-1, keepdims=True)).astype(np.float32)
            den = e.sum(-1, keepdims=True, dtype=np.float32)
            num = bf16_round(e).astype(np.float32)
            o = np.einsum("blp,bpd->bld", num, V.astype(np.float32))
            out[:, h] = (o / den).astype(np.float64)
        return out

    def layer_step(self, x, li, nb, L, P, cache):
        cfg = self.cfg
        Hq, Hkv, d = cfg["heads"], cfg["kv_heads"], cfg["head_dim"]
        ang = rope_angles(np.arange(P, P + L), d, cfg["rope_theta"])
        w = self.layer(li)
        h = bf16_round(norm32(x, w["ln1"], cfg["rms_eps"]))
        q, k, v = mm32(h, w["wq"].T), mm32(h, w["wk"].T), mm32(h, w["wv"].T)
        if cfg["qkv_bias"]:
            q, k, v = q + w["bq"], k + w["bk"], v + w["bv"]
        q = bf16_round(apply_rope(q.reshape(nb, L, Hq, d).transpose(0, 2, 1, 3), ang))
        k = bf16_round(apply_rope(k.reshape(nb, L, Hkv, d).transpose(0, 2, 1, 3), ang))
        v = bf16_round(v.reshape(nb, L, Hkv, d).transpose(0, 2, 1, 3))
        o = self.attention32(q, k, v, cache.k[li, :, :P], cache.v[li, :, :P])
        o = bf16_round(o.transpose(0, 2, 1, 3).reshape(nb, L, Hq * d))
        x = (x.astype(np.float32) + mm32(o, w["wo"].T).astype(np.float32)).astype(np.float64)
        h2 = bf16_round(norm32(x, w["ln2"], cfg["rms_eps"]))
        g = mm32(h2, w["w_gate"].T).astype(np.float32)
        u = mm32(h2, w["w_up"].T).astype(np.float32)
        a = bf16_round((g / (np.float32(1) + np.exp(-g)) * u).astype(np.float64))
        return (x.astype(np.float32) + mm32(a, w["w_down"].T).astype(np.float32)).astype(np.float64)

    def forward32(self, tokens, P, cache):
        """conf, pred, final residual stream of the branches tokens [nb, L]."""
        tokens = np.asarray(tokens)
        nb, L = tokens.shape
        x = self.embed[tokens]
        for li in range(self.cfg["layers"]):
            x = self.layer_step(x, li, nb, L, P, cache)
        hf = bf16_round(norm32(x, self.final_norm, self.cfg["rms_eps"]))
        conf, pred = confidence(mm32(hf, self.lm_head.T), self.cfg["mask_id"])
        return conf, pred, x
