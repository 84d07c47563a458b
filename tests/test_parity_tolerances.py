"""The fixed tolerances of the GPU parity tests (gpu_util) hold for an
independent correct bf16 computation of the verify forward (bf16_variant: the
oracle's rounding points, float32 arithmetic between them) on the parity
models, so they demand no more than bf16 arithmetic allows:
  * each layer fed the same input: rel-L2 within LAYER_TOL of the faithful
    oracle and LAYER_TOL_PURE of the pure one;
  * the oracle's LM head on the variant's own final rows: the same confidences
    within TF_CONF_TOL and the same candidates at margins >= NEAR_TIE;
  * end to end: confidences within conf_tol(cfg) of the pure oracle.
It also records what they cannot demand: end to end, a few candidate tokens
with margins above 1e-3 differ from the faithful oracle's (two bf16
computations part at that level after a few layers), so end-to-end integer
decisions are compared teacher-forced at the decision."""
import numpy as np
import pytest

import synth
from bf16_variant import Bf16Variant
from gpu_util import (LAYER_TOL, LAYER_TOL_PURE, NEAR_TIE, TF_CONF_TOL, conf_tol, logit_std,
                      rel_l2, vocab_margin)
from oracle import KVCache, OracleModel, lopa

CASES = [("tiny", 64, 16, 3), ("small", 100, 32, 7), ("small", 37, 32, 15), ("small128", 40, 16, 2)]


@pytest.mark.parametrize("cfgname,P,L,k", CASES)
def test_tolerances_hold_for_an_independent_bf16_forward(cfgname, P, L, k):
    cfg = synth.config(cfgname)
    w = synth.to_bf16_values(synth.model_weights(cfg))
    faith, pure, var = OracleModel(cfg, w, "faithful"), OracleModel(cfg, w, "pure"), Bf16Variant(cfg, w)
    cache = KVCache(cfg, P + L)
    lopa.prefill(faith, cache, synth.prompt(cfg, P).numpy(), L)
    rng = np.random.default_rng(P + L + k)
    mask, nb = cfg["mask_id"], k + 1
    bt = np.where(rng.random((nb, L)) < 0.7, mask, rng.integers(0, cfg["vocab"] - 1, (nb, L)))
    bt[0] = mask
    x = faith.embed[bt]
    for li in range(cfg["layers"]):
        xv = var.layer_step(x, li, nb, L, P, cache)
        of = faith.forward_block(bt, P, cache, x_in=x, first_layer=li, n_layers=li + 1)["x"]
        op = pure.forward_block(bt, P, cache, x_in=x, first_layer=li, n_layers=li + 1)["x"]
        assert rel_l2(xv, of) <= LAYER_TOL and rel_l2(xv, op) <= LAYER_TOL_PURE
        x = xv
    conf, pred, x_last = var.forward32(bt, P, cache)
    tf = faith.lm_from_residual(x_last)
    dec = vocab_margin(tf["logits"], mask) >= NEAR_TIE
    assert np.max(np.abs(conf - tf["conf"])) <= TF_CONF_TOL
    assert np.array_equal(pred[dec], tf["pred"][dec])
    e_pure = np.max(np.abs(conf - pure.forward_block(bt, P, cache)["conf"]))
    rf = faith.forward_block(bt, P, cache, keep_hidden=True)
    dec_e = vocab_margin(rf["logits"], mask) >= NEAR_TIE
    print(f"{cfgname}: logit std {logit_std(cfg):.1f}, end to end |conf - pure| {e_pure:.2e} "
          f"(tolerance {conf_tol(cfg):.2e}), {int(np.sum(pred[dec_e] != rf['pred'][dec_e]))} "
          f"decided candidates differ from the faithful oracle end to end")
    assert e_pure <= conf_tol(cfg)
