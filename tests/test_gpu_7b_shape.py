"""GPU parity at the full model shapes of the measured workloads, in the launch
configuration bench.py times (every plan and kernel of the step at that size):
  * Dream-7B, prefix 512, k = 7 (8 branches x 32 rows: one 256-row tile);
  * Dream-7B, prefix 2048, k = 15 (16 branches x 32 rows: two row tiles);
  * LLaDA-8B (MHA, no biases), prefix 1024, k = 7.

One whole LoPA iteration (Alg. 1) at each shape, all layers, every row:
  * the block's initial forward (all positions masked) gives the state; its
    confidences / candidates against the oracle's LM head on its final rows;
  * lopa_build_branches on that state against the oracle's Eq. 1 / top-k on
    the same confidences (bit-exact);
  * lopa_verify_forward of all k+1 branches against the float64 oracle with
    the fixed tolerances of gpu_util.check_forward: every layer (every seventh
    and the last at prefix 2048) fed the GPU's own input residual stream
    (rel-L2 vs the bf16-faithful layer), confidences
    within 2e-2 of the pure oracle end to end, and the oracle's LM head +
    softmax on the GPU's own final rows (confidence within 1e-3, candidate
    tokens equal where the top-2 margin is >= 1e-3);
  * lopa_branch_confidence_select against Eq. 2 on the GPU's confidences;
  * lopa_commit_kv: the cache rows equal the winner's staged K/V bit for bit.
The prefix K/V are the GPU's own block-causal prefill, read back and handed to
the oracle (teacher-forced prefix). The oracle streams the weights layer by
layer from the GPU's bf16 tensors. The LM head is spread (N(0, 5/sqrt(H)): logit std 5)
so that confidences are informative."""
import types

import numpy as np
import pytest
import torch

import synth
from gpu_util import (NEAR_TIE, check_forward, conf_tol, f32, gpu_residual, log, score_margin,
                      tf_lm_check)
from oracle import KVCache, OracleModel, lopa

pytestmark = pytest.mark.gpu

L = 32
TAU = 0.9
CASES = [("dream7b_spread", 512, 7), ("dream7b_spread", 2048, 15), ("llada8b_spread", 1024, 7)]


class _Layers:
    """The oracle's view of the GPU's bf16 layer weights, one layer at a time."""

    def __init__(self, w):
        self.w = w

    def __len__(self):
        return len(self.w["layers"])

    def __getitem__(self, i):
        return {k: v.float().cpu() for k, v in self.w["layers"][i].items()}


@pytest.fixture(scope="module", params=CASES, ids=lambda c: f"{c[0]}-P{c[1]}-k{c[2]}")
def big(request):
    import paper_2512_16229_amd as lp
    name, P, K = request.param
    log(f"full shape {name}: prefix {P}, k {K}")
    cfg = synth.config(name)
    w = synth.model_weights(cfg, device="cuda", dtype=torch.bfloat16)
    model = lp.Model(cfg, w)
    kv = lp.KV(model, P + L, K + 1, L)
    dec = lp.Decoder(model, kv, L, K, TAU)
    assert dec.prefill(synth.prompt(cfg, P, device="cuda")) == P
    torch.cuda.synchronize()
    host = {"embed": w["embed"].float().cpu(), "layers": _Layers(w),
            "final_norm": w["final_norm"].float().cpu(), "lm_head": w["lm_head"].float().cpu()}
    cache = KVCache(cfg, P + L)
    for layer in range(cfg["layers"]):
        kg, vg = kv.read(layer, 0, P)
        cache.k[layer, :, :P] = kg.float().cpu().numpy()
        cache.v[layer, :, :P] = vg.float().cpu().numpy()
    s = types.SimpleNamespace(lp=lp, cfg=cfg, model=model, kv=kv, P=P, L=L, k=K, dec=dec,
                              cache_f=cache)
    # one converted layer at a time, shared by both modes (bf16-valued weights)
    s.faith = OracleModel(cfg, host, "faithful", keep_layers=1, bf16_weights=True)
    s.pure = OracleModel(cfg, host, "pure", keep_layers=1, share=s.faith,
                         bf16_weights=True)
    yield s
    del s, dec, kv, model, w, host
    torch.cuda.empty_cache()


def test_lopa_iteration_full_depth(big):
    s = big
    lp, cfg, P, K = s.lp, s.cfg, s.P, s.k
    mask, nb = cfg["mask_id"], K + 1
    dec = s.dec
    # the block's initial forward: the state of the first iteration
    dec.init_block(P)
    tokens = dec.tokens.cpu().numpy()
    conf0 = dec.conf.cpu().numpy().astype(np.float64)
    pred0 = dec.pred.cpu().numpy()
    log(f"  initial forward: conf {conf0.min():.3f}..{conf0.max():.3f}")
    tf_lm_check(s, gpu_residual(s, tokens[None], cfg["layers"]), conf0[None], pred0[None],
                "initial forward")
    # Eq. 1 + lookahead branches (Alg. 1 steps 1-2) on that state
    lp.lopa_build_branches(dec.tokens, dec.conf, dec.pred, L, mask, TAU, K, dec.branch_tokens,
                           dec.fill_pos, dec.valid, dec.n_valid)
    bt = dec.branch_tokens.view(nb, L).cpu().numpy()
    rbt, rfp, rva, rnv = lopa.build_branches(tokens, conf0, pred0, mask, f32(TAU), K)
    assert np.array_equal(bt, rbt) and np.array_equal(dec.valid.cpu().numpy(), rva)
    assert int(dec.n_valid.item()) == rnv
    # the verify forward of all branches (Alg. 1 step 3), every layer
    lp.lopa_verify_forward(s.model, s.kv, P, dec.branch_tokens, nb, L, dec.conf_b, dec.pred_b)
    gc = dec.conf_b.view(nb, L).cpu().numpy().astype(np.float64)
    gp = dec.pred_b.view(nb, L).cpu().numpy()
    log(f"  verify forward: {nb * L} rows, conf {gc.min():.3f}..{gc.max():.3f}")
    # every layer teacher-forced at the two shorter prefixes; at prefix 2048 (the
    # oracle's attention over 2080 keys for 512 rows dominates the test's time)
    # every seventh layer and the last, and the end-to-end sweeps over all
    tf_layers = True if P <= 1024 else list(range(0, cfg["layers"], 7)) + [cfg["layers"] - 1]
    st = check_forward(s, rbt, gc, gp, layers=tf_layers, e2e_faithful=True, label="verify forward")
    # Eq. 2 on the GPU's confidences, and vs the pure oracle's scores
    outs = (dec.scores, dec.winner, dec.next_tokens, dec.next_conf, dec.next_pred,
            dec.next_unfilled)
    lp.lopa_branch_confidence_select(dec.branch_tokens, dec.conf_b, dec.pred_b, dec.valid, nb, L,
                                     mask, *outs)
    gs = dec.scores.cpu().numpy().astype(np.float64)
    ts, tw = lopa.select(rbt, gc, rva, mask)
    ps, _ = lopa.select(rbt, st["pure"]["conf"], rva, mask)
    fin = np.isfinite(ts)
    assert np.max(np.abs(gs[fin] - ts[fin]), initial=0) <= 1e-5
    assert np.max(np.abs(gs[fin] - ps[fin]), initial=0) <= conf_tol(s.cfg)
    w = int(dec.winner.item())
    if score_margin(ts) >= NEAR_TIE:
        assert np.array_equal(rbt[w], rbt[tw])
    assert np.array_equal(dec.next_tokens.cpu().numpy(), rbt[w])
    assert np.array_equal(dec.next_conf.cpu().numpy(), dec.conf_b.view(nb, L)[w].cpu().numpy())
    # commit the winner's K/V (Sec. 3.4): the cache rows equal its staging
    lp.lopa_commit_kv(s.kv, dec.winner, P, L, dec.append_offset)
    assert int(dec.append_offset.item()) == P
    for layer in (0, cfg["layers"] // 2, cfg["layers"] - 1):
        kc, vc = s.kv.read(layer, P, L)
        ks, vs = s.kv.read_staging(w, layer, L)
        assert torch.equal(kc, ks) and torch.equal(vc, vs)
    log(f"  winner {w}, score margin {score_margin(ts):.2e}")
