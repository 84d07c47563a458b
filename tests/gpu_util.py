"""Helpers shared by the GPU parity tests (inputs, oracle runs, near-tie margins)."""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import KVCache, OracleModel, lopa

# Fixed tolerances of the GPU parity tests (none depends on a measured GPU
# error; the derivation of each is in the design notes, reading R24):
NEAR_TIE = 1e-3      # an integer decision may differ only where the oracle's own margin
                     # (top-2 probability gap, |conf - tau|, top-k gap, score gap) is below this
CONF_TOL = 2e-2      # end to end: |GPU conf / Eq. 2 score - pure float64 oracle|, same inputs
                     # (bf16-valued weights, tokens, prefix K/V), for LM heads whose logit
                     # std sigma is <= 5; conf_tol(cfg) scales it by sigma / 5 above that
TF_CONF_TOL = 1e-4   # |GPU conf - the oracle's LM head + softmax on the GPU's own final
                     # residual rows| (only the LM head's float32 sums differ, ~1e-5;
                     # a final normed value at a bf16 midpoint may round either way)
TF_CONF_TOL_FP8 = 5e-4  # the same for the FP8 LM head (per-row and per-column scales)
BF16_TIE_REL = 2.0 ** -20  # float32 distance of the GPU's RMSNorm from the exact value
LAYER_TOL = 1e-2     # one layer fed the GPU's input: rel-L2 of the GPU's output residual
                     # stream vs the bf16-faithful oracle layer
LAYER_TOL_PURE = 2e-2  # the same vs the pure float64 layer
LAYER_TOL_FP8 = 5e-2   # the FP8 modes' layer vs the oracle's FP8 mode (E4M3 codes of the
                       # GEMM operands flip where bf16-level differences meet a rounding midpoint)


def logit_std(cfg) -> float:
    """Standard deviation of the synthetic model's logits: lm_std * sqrt(hidden)."""
    return float(cfg["lm_std"]) * float(np.sqrt(cfg["hidden"]))


def conf_tol(cfg) -> float:
    """End-to-end confidence tolerance of a model: CONF_TOL, scaled by sigma / 5
    for logit std sigma > 5. A confidence moves by about p (1 - p) times the
    logit change, and bf16 rounding changes the final rows by a fixed relative
    amount, so the bf16-vs-float64 difference grows in proportion to sigma
    (tests/test_parity_tolerances.py measures it on an independent bf16
    computation: within 2e-2 at sigma 5, up to about 2.6e-2 at sigma 8)."""
    return CONF_TOL * max(1.0, logit_std(cfg) / 5.0)


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
        # the pure oracle gets the same bf16-valued weights the GPU streams (the
        # faithful modes round them anyway): weight rounding is not part of the
        # arithmetic being compared
        self.pure = OracleModel(self.cfg, synth.to_bf16_values(self.w), "pure")
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


def rel_l2(a, b) -> float:
    return float(np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(b), 1e-300))


def gpu_residual(s, branch_tokens: np.ndarray, n_layers: int, P=None) -> np.ndarray:
    """The GPU's fp32 residual stream after n_layers layers (lopa_debug_hidden)."""
    P = s.P if P is None else P
    nb, L = branch_tokens.shape
    x = torch.empty(nb * L * s.cfg["hidden"], dtype=torch.float32, device="cuda")
    bt = torch.tensor(branch_tokens, dtype=torch.int32, device="cuda").reshape(-1)
    s.lp.lopa_debug_hidden(s.model, s.kv, P, bt, nb, L, n_layers, x)
    torch.cuda.synchronize()
    return x.view(nb, L, -1).cpu().numpy().astype(np.float64)


def _full_size(cfg):
    """The 7B / 8B shapes (billions of weights): the oracle runs them layer by
    layer, without a second whole-forward pass."""
    return cfg["layers"] * cfg["hidden"] ** 2 >= 1e8


def check_forward(s, bt, conf_g, pred_g, P=None, cache_f=None, cache_p=None, causal_blk=0,
                  layers=True, label="", e2e_faithful=True):
    """The parity protocol of one verify forward whose prefix K/V the GPU shares
    with the faithful oracle (teacher-forced prefix; cache_f holds those rows):

      * end to end: |GPU conf - pure oracle conf| <= conf_tol(cfg) (the pure
        oracle on the same prefix K/V values, cache_p; default cache_f), on
        cases where the faithful oracle itself is within that of the pure one
        (e2e_faithful; at the full model depths bf16 rounding alone moves the
        confidences by more, and only the teacher-forced checks apply);
      * per layer (layers=True): each layer of the faithful and the pure oracle
        fed the GPU's own input residual stream; the GPU's output within
        LAYER_TOL / LAYER_TOL_PURE rel-L2;
      * decisions: the faithful oracle's LM head + softmax on the GPU's own
        final residual rows (tf_lm_check): GPU conf within TF_CONF_TOL and
        every candidate token whose oracle margin is >= NEAR_TIE identical;
      * logged, not asserted (e2e_faithful): candidate tokens that differ from
        the end-to-end faithful oracle at margins >= NEAR_TIE (two bf16
        computations that sum in a different order part at that level after a
        few layers).
    FP8 model modes go to check_forward_fp8. Returns a dict of the figures."""
    if getattr(s.faith, "fp8_mlp", False):
        return check_forward_fp8(s, bt, conf_g, pred_g, P, cache_f, causal_blk, layers, label)
    return _check_forward_bf16(s, bt, conf_g, pred_g, P, cache_f, cache_p, causal_blk, layers,
                               label, e2e_faithful)


def _check_forward_bf16(s, bt, conf_g, pred_g, P, cache_f, cache_p, causal_blk, layers, label,
                        e2e_faithful):
    """The bf16 protocol of check_forward (see there), in one sweep over the
    layers (each layer's weights are used by every comparison before the next
    layer's are converted); every figure is logged before the asserts."""
    P = s.P if P is None else P
    cache_f = s.cache_f if cache_f is None else cache_f
    cache_p = cache_f if cache_p is None else cache_p
    mask, Ly = s.cfg["mask_id"], s.cfg["layers"]
    big = _full_size(s.cfg)   # full-size shapes: a progress line per layer

    def one(model, x, li, cache):
        return model.forward_block(bt, P, cache, x_in=x, first_layer=li, n_layers=li + 1,
                                   causal_blk=causal_blk)["x"]

    # layers: True (all), a list of layer indices, or False
    which = set(range(Ly)) if layers is True else (set(layers) if layers else set())
    rel_f, rel_p = [], []
    x0 = s.faith.embed[np.asarray(bt)]
    x_g, g_at = x0, 0              # a GPU residual stream and the layers it has passed
    x_p, x_f = x0, x0              # pure and faithful end to end
    for li in range(Ly):
        if li in which:
            x_in = x_g if g_at == li else gpu_residual(s, bt, li, P)
            xg = gpu_residual(s, bt, li + 1, P)
            rel_f.append(rel_l2(xg, one(s.faith, x_in, li, cache_f)))
            rel_p.append(rel_l2(xg, one(s.pure, x_in, li, cache_f)))
            x_g, g_at = xg, li + 1
        x_p = one(s.pure, x_p, li, cache_p)
        if e2e_faithful:
            x_f = one(s.faith, x_f, li, cache_f)
        if big:
            tf = li in which
            log(f"    layer {li}: teacher-forced rel-L2 vs faithful "
                f"{rel_f[-1] if tf else 0:.2e}, vs pure {rel_p[-1] if tf else 0:.2e}; end "
                f"to end: gpu-pure {rel_l2(x_g, x_p) if tf else 0:.2e}, faithful-pure "
                f"{rel_l2(x_f, x_p) if e2e_faithful else 0:.2e}")
    x_last = x_g if g_at == Ly else gpu_residual(s, bt, Ly, P)
    rp = s.pure.lm_from_residual(x_p)
    e_pure = float(np.max(np.abs(conf_g - rp["conf"])))
    rf_e2e, bad_e2e, e_faith, n_dec, e_bf16 = None, -1, float("nan"), 0, 0.0
    if e2e_faithful:
        out = s.faith.lm_from_residual(x_f)
        e_bf16 = float(np.max(np.abs(out["conf"] - rp["conf"])))   # bf16 vs float64, no GPU
        rf_e2e = {"conf": out["conf"], "pred": out["pred"], "logits": out["logits"],
                  "hidden": out["hidden"]}
        # the block K/V of every layer, as forward_block returns them
        full = s.faith.forward_block(bt, P, cache_f, causal_blk=causal_blk) if not big else None
        if full is not None:
            rf_e2e["k"], rf_e2e["v"] = full["k"], full["v"]
        dec_e = vocab_margin(out["logits"], mask) >= NEAR_TIE
        bad_e2e, n_dec = int(np.sum(pred_g[dec_e] != out["pred"][dec_e])), int(dec_e.sum())
        e_faith = float(np.max(np.abs(conf_g - out["conf"])))
    log(f"  {label} conf: gpu-pure {e_pure:.2e} gpu-faithful {e_faith:.2e} faithful-pure "
        f"{e_bf16:.2e} | per-layer rel-L2 "
        f"vs faithful {' '.join(f'{v:.1e}' for v in rel_f)} vs pure "
        f"{' '.join(f'{v:.1e}' for v in rel_p)} | end-to-end faithful: {bad_e2e}/{n_dec} decided "
        f"tokens differ")
    e_tf, n_excused, n_ties = tf_lm_check(s, x_last, conf_g, pred_g, label)
    log(f"  {label} LM head on the GPU's rows: dconf {e_tf:.1e}, {n_excused} near-ties excused, "
        f"{n_ties} rows through a bf16 midpoint")
    # end-to-end confidences: within the tolerance, unless the bf16 arithmetic
    # itself (the faithful oracle, no GPU) is farther than that from float64
    # on this case; then only the teacher-forced decisions above decide
    tol = conf_tol(s.cfg)
    if e_bf16 <= tol:
        assert e_pure <= tol, f"{label}: |conf - pure| = {e_pure:.3e} > {tol:.3e}"
    else:
        log(f"  {label}: bf16 arithmetic alone differs from float64 by {e_bf16:.2e} > {tol:.2e}; "
            f"end-to-end confidences not bounded on this case")
    for li, rf, rpu in zip(sorted(which), rel_f, rel_p):
        assert rf <= LAYER_TOL, f"{label}: layer {li} rel-L2 vs faithful {rf:.2e} > {LAYER_TOL}"
        assert rpu <= LAYER_TOL_PURE, f"{label}: layer {li} rel-L2 vs pure {rpu:.2e}"
    assert not np.any(pred_g == mask)
    return dict(e_pure=e_pure, e_faith=e_faith, e_bf16=e_bf16, e_tf=e_tf,
                worst_f=max(rel_f, default=0.0),
                worst_p=max(rel_p, default=0.0), excused=n_excused, bad_e2e=bad_e2e,
                faith=rf_e2e, pure=rp)


def e4m3_tie_rows(h) -> np.ndarray:
    """Rows of h [..., K] with a value within float32 distance of an E4M3
    rounding midpoint after the per-row scaling (such a code is decided either
    way by float32 vs float64 arithmetic; both are the rule)."""
    from oracle.fp8 import E4M3_MAX, e4m3_round
    v = np.abs(h) * (E4M3_MAX / np.max(np.abs(h), axis=-1, keepdims=True))
    return ~np.all(e4m3_round(v * (1 - 1e-5)) == e4m3_round(v * (1 + 1e-5)), axis=-1)


def check_forward_fp8(s, bt, conf_g, pred_g, P=None, cache_f=None, causal_blk=0, layers=True,
                      label=""):
    """The FP8 modes against the oracle's FP8 mode of the same name (the same
    quantisation points and rules): the layers (all, or the listed indices)
    fed the GPU's own input within LAYER_TOL_FP8 rel-L2, and the oracle's LM
    head on the GPU's own final rows (FP8 in the "fp8" mode) within
    TF_CONF_TOL_FP8 with identical candidates at margins >= NEAR_TIE, on the
    rows whose final normed values have no E4M3 tie; end to end the
    confidences are logged (E4M3 code changes upstream move them by more than
    the bf16 tolerance)."""
    from oracle.model import rms_norm
    P = s.P if P is None else P
    cache_f = s.cache_f if cache_f is None else cache_f
    mask, Ly = s.cfg["mask_id"], s.cfg["layers"]
    which = list(range(Ly)) if layers is True else (list(layers) if layers else [])
    big = _full_size(s.cfg)
    rels = []
    for li in which:
        x_in = s.faith.embed[np.asarray(bt)] if li == 0 else gpu_residual(s, bt, li, P)
        xg = gpu_residual(s, bt, li + 1, P)
        of = s.faith.forward_block(bt, P, cache_f, x_in=x_in, first_layer=li, n_layers=li + 1,
                                   causal_blk=causal_blk)["x"]
        rels.append(rel_l2(xg, of))
        if big:
            log(f"    layer {li}: rel-L2 vs the FP8 oracle {rels[-1]:.2e}")
    x_last = gpu_residual(s, bt, Ly, P)
    rf, e_e2e = None, float("nan")
    if not big:
        rf = s.faith.forward_block(bt, P, cache_f, keep_hidden=True, causal_blk=causal_blk)
        e_e2e = float(np.max(np.abs(conf_g - rf["conf"])))
    if s.faith.fp8_qkv_lm:
        # FP8 LM head: rows with an E4M3 tie in their final normed values are
        # left out (either code is a correct rounding)
        tf = s.faith.lm_from_residual(x_last)
        ties = e4m3_tie_rows(rms_norm(x_last, s.faith.final_norm, s.cfg["rms_eps"]))
        ok = ~ties
        e_tf = float(np.max(np.abs(conf_g - tf["conf"])[ok], initial=0.0))
        dec = (vocab_margin(tf["logits"], mask) >= NEAR_TIE) & ok
        bad = int(np.sum(pred_g[dec] != tf["pred"][dec]))
        lm = (f"dconf {e_tf:.1e}, {int(ties.sum())} rows with E4M3 ties, "
              f"{int((~dec & ok).sum())} near-ties")
    else:
        lm = None
    log(f"  {label} fp8: layer rel-L2 {' '.join(f'{v:.1e}' for v in rels)} | LM head on GPU rows: "
        f"{lm if lm else 'bf16 (below)'} | end to end |conf - fp8 oracle| {e_e2e:.2e}")
    for li, r in zip(which, rels):
        assert r <= LAYER_TOL_FP8, f"{label}: layer {li} rel-L2 vs the FP8 oracle {r:.2e}"
    if lm is None:
        # the bf16 LM head of the MLP-only mode: the bf16 protocol, with its
        # enumeration of the rows whose normed values sit at a bf16 midpoint
        e_tf, n_excused, n_ties = tf_lm_check(s, x_last, conf_g, pred_g, label)
        log(f"  {label} LM head (bf16) on the GPU's rows: dconf {e_tf:.1e}, {n_excused} near-ties "
            f"excused, {n_ties} rows through a bf16 midpoint")
        bad = 0
    assert e_tf <= TF_CONF_TOL_FP8, f"{label}: |conf - oracle LM head on GPU rows| = {e_tf:.2e}"
    assert bad == 0, f"{label}: {bad} decided candidate tokens differ (teacher-forced LM head)"
    assert not np.any(pred_g == mask)
    return dict(worst_f=max(rels, default=0.0), e_tf=e_tf, e_e2e=e_e2e, faith=rf)


def tf_lm_check(s, x_last, conf_g, pred_g, label=""):
    """The faithful oracle's final RMSNorm + LM head + softmax (Sec. 3.1) on the
    GPU's own final residual rows x_last: the GPU's confidences within
    TF_CONF_TOL and its candidates equal wherever the oracle's top-2 margin is
    >= NEAR_TIE. A normed value within float32 distance of a bf16 rounding
    midpoint may be rounded either way by a correct implementation: a row
    that misses with the oracle's rounding is accepted if it matches with the
    other rounding of some of its tied values (all combinations, at most 2^10).
    Returns (max conf difference of the accepted rows, near-ties excused, rows
    accepted through a tie)."""
    from oracle.model import bf16_round, confidence, rms_norm
    mask = s.cfg["mask_id"]
    tf = s.faith.lm_from_residual(x_last)
    conf_o, pred_o, logits = tf["conf"], tf["pred"], tf["logits"]
    marg = vocab_margin(logits, mask)
    err = np.abs(conf_g - conf_o)
    ok = (err <= TF_CONF_TOL) & ((marg < NEAR_TIE) | (pred_g == pred_o))
    n_excused = int(np.sum(marg < NEAR_TIE))
    worst = float(np.max(err[ok], initial=0.0))
    bad = np.argwhere(~ok)
    n_ties = 0
    if bad.size:
        x2 = np.asarray(x_last).reshape(-1, x_last.shape[-1])
        hf = rms_norm(x2, s.faith.final_norm, s.cfg["rms_eps"])
        base = tf["hidden"].reshape(-1, x2.shape[-1])
        lo, hi = bf16_round(hf * (1 - BF16_TIE_REL)), bf16_round(hf * (1 + BF16_TIE_REL))
        W = s.faith.lm_head
        shp = conf_g.shape
        for idx in bad:
            idx = tuple(idx)
            r = int(np.ravel_multi_index(idx, shp))
            ties = np.flatnonzero(lo[r] != hi[r])
            assert 0 < ties.size <= 10, (f"{label}: row {idx}: conf {conf_g[idx]:.6f} vs "
                                         f"{conf_o[idx]:.6f}, pred {pred_g[idx]} vs {pred_o[idx]}, "
                                         f"{ties.size} values at a midpoint")
            alt = np.where(base[r, ties] == lo[r, ties], hi[r, ties], lo[r, ties]) - base[r, ties]
            dl = W[:, ties] * alt                                   # [V, n] logit changes
            lg0 = logits.reshape(-1, logits.shape[-1])[r]
            found = False
            for sub in range(1, 1 << ties.size):
                pick = np.array([(sub >> i) & 1 for i in range(ties.size)], dtype=np.float64)
                lg = lg0 + dl @ pick
                c, p = confidence(lg[None], mask)
                m = vocab_margin(lg[None], mask)[0]
                e = abs(conf_g[idx] - c[0])
                if e <= TF_CONF_TOL and (m < NEAR_TIE or pred_g[idx] == p[0]):
                    found, worst = True, max(worst, e)
                    break
            assert found, f"{label}: row {idx} matches no rounding of its tied values"
            n_ties += 1
    return worst, n_excused, n_ties
