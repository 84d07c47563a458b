"""Helpers shared by the GPU parity tests (inputs, oracle runs, near-tie margins)."""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import KVCache, OracleModel, lopa

NEAR_TIE = 1e-3     # integer decisions closer than this (in probability units) may differ
CONF_TOL = 2e-2     # abs tolerance of confidences and branch scores (bf16 path vs float64)
# GPU vs the oracle that rounds at the same points. The two differ only by fp32 vs
# fp64 summation, but that flips a few bf16 roundings per layer (hidden-state
# rel-L2 ~1e-3 after two layers) which the LM head amplifies by its logit scale;
# their confidence gap is bounded like the bf16 error itself (conf_tolerance).
FAITHFUL_TOL = 2e-2


def faithful_bound(bf16_own_error: float) -> float:
    """Bound on |GPU - bf16-faithful oracle| for confidences.

    Both are bf16 computations with the same rounding points that round in a
    different order (fp32 vs fp64 sums; a running vs a global softmax maximum),
    so each sits at about the bf16 distance e from the exact float64 result,
    e = |faithful - float64| measured on the case itself (no GPU involved).
    Bound: 2e, and never below the 2e-2 confidence tolerance."""
    return max(CONF_TOL, 2.0 * bf16_own_error)


def conf_tolerance(bf16_own_error: float) -> float:
    """Bound on |GPU - float64 oracle| (the bf16 result vs the exact one): 2e-2,
    or twice the faithful oracle's own bf16 distance where that is larger."""
    return max(CONF_TOL, 2.0 * bf16_own_error)


def near_tie(eps: float) -> float:
    """Margin below which an integer decision may differ between the GPU and the
    bf16-faithful oracle: 1e-3, or twice the measured confidence gap eps of the
    two computations (a top-2 pair whose members each move by up to eps can swap
    only if they are within 2 eps). eps itself is asserted to stay within
    conf_tolerance of the case."""
    return max(NEAR_TIE, 2.0 * eps)


def log(msg: str):
    print(msg, flush=True)


def to_dev_bf16(w):
    if isinstance(w, dict):
        return {k: to_dev_bf16(v) for k, v in w.items()}
    if isinstance(w, list):
        return [to_dev_bf16(v) for v in w]
    return w.to(device="cuda", dtype=torch.bfloat16).contiguous()


def f32(x: float) -> float:
    """The fp32 value of x, as the GPU compares with it."""
    return float(np.float32(x))


class Setup:
    """Same seeded model + prompt on both sides, each side prefilled by itself."""

    def __init__(self, cfgname: str, P: int, L: int, k: int, max_len=None, precision="bf16",
                 **over):
        """precision "fp8_mlp" / "fp8": the GPU model's MLP (and QKV and LM head)
        in FP8, and self.faith the oracle's mode of the same name (the same
        quantisation points)."""
        import paper_2512_16229_amd as lp
        self.lp = lp
        self.cfg = synth.config(cfgname, **over)
        self.w = synth.model_weights(self.cfg)
        self.P, self.L, self.k = P, L, k
        self.max_len = max_len or (P + 2 * L)
        self.model = lp.Model(self.cfg, to_dev_bf16(self.w), precision=precision)
        self.kv = lp.KV(self.model, self.max_len, k + 1, L)
        self.prompt = synth.prompt(self.cfg, P)
        self.pure = OracleModel(self.cfg, self.w, "pure")
        self.faith = OracleModel(self.cfg, self.w, "faithful" if precision == "bf16" else precision)
        self.cache_p = KVCache(self.cfg, self.max_len)
        self.cache_f = KVCache(self.cfg, self.max_len)
        if P:
            lopa.prefill(self.pure, self.cache_p, self.prompt.numpy(), L)
            lopa.prefill(self.faith, self.cache_f, self.prompt.numpy(), L)

    def gpu_prefill(self, tau=0.9):
        dec = self.lp.Decoder(self.model, self.kv, self.L, self.k, tau)
        if self.P:
            assert dec.prefill(self.prompt) == self.P
        return dec

    def load_oracle_cache(self, upto=None):
        """Teacher forcing of the prefix: write the bf16-faithful oracle's cache rows
        [0, upto) into the GPU cache (their values are exact bf16 numbers)."""
        upto = self.P if upto is None else upto
        if upto == 0:
            return
        for layer in range(self.cfg["layers"]):
            k = torch.tensor(self.cache_f.k[layer, :, :upto], dtype=torch.bfloat16, device="cuda")
            v = torch.tensor(self.cache_f.v[layer, :, :upto], dtype=torch.bfloat16, device="cuda")
            self.kv.write(layer, 0, k.contiguous(), v.contiguous())
        torch.cuda.synchronize()

    def gpu_forward(self, branch_tokens: np.ndarray, P=None):
        P = self.P if P is None else P
        nb, L = branch_tokens.shape
        bt = torch.tensor(branch_tokens, dtype=torch.int32, device="cuda").reshape(-1)
        conf = torch.empty(nb * L, dtype=torch.float32, device="cuda")
        pred = torch.empty(nb * L, dtype=torch.int32, device="cuda")
        self.lp.lopa_verify_forward(self.model, self.kv, P, bt, nb, L, conf, pred)
        torch.cuda.synchronize()
        return conf.view(nb, L).cpu().numpy().astype(np.float64), pred.view(nb, L).cpu().numpy()


def vocab_margin(logits: np.ndarray, mask_id: int) -> np.ndarray:
    """p1 - p2 of the softmax without the mask token (oracle precision)."""
    lg = np.array(logits, dtype=np.float64, copy=True)
    lg[..., mask_id] = -np.inf
    p = np.exp(lg - lg.max(-1, keepdims=True))
    p /= p.sum(-1, keepdims=True)
    top2 = np.sort(p, axis=-1)[..., -2:]
    return top2[..., 1] - top2[..., 0]


def build_margin(tokens, conf, mask_id, tau, k, n_eligible=None) -> float:
    """Smallest confidence gap that decides lopa_build_branches' output
    (n_eligible: the fallback and the lookahead fills only below it)."""
    tokens, conf = np.asarray(tokens), np.asarray(conf, dtype=np.float64)
    n_el = len(tokens) if n_eligible is None else n_eligible
    M = np.flatnonzero(tokens == mask_id)
    if M.size == 0:
        return np.inf
    gaps = [np.min(np.abs(conf[M] - tau))]
    Me = M[M < n_el]
    c = np.sort(conf[Me])[::-1]
    if not np.any(conf[M] > tau) and c.size > 1:
        gaps.append(c[0] - c[1])
    fill = lopa.threshold_fill(conf, tokens == mask_id, tau, n_eligible)
    rem = np.setdiff1d(Me, fill)
    cr = np.sort(conf[rem])[::-1]
    if 0 < k < cr.size:
        gaps.append(cr[k - 1] - cr[k])
    return float(min(gaps))


def score_margin(scores) -> float:
    s = np.sort(np.asarray(scores, dtype=np.float64)[np.isfinite(scores)])[::-1]
    if np.any(np.isposinf(scores)):
        return np.inf
    return float(s[0] - s[1]) if s.size > 1 else np.inf
