"""GPU parity of the FP8 model mode (LOPA_PRECISION_FP8: QKV, O, gate / up /
down and the LM head in W8A8 E4M3) at the full Dream-7B shape, prefix 512, k = 7,
in the launch configuration bench.py times for its FP8 step figure, at prefix
2048, k = 15 (two row tiles, the grouped attention form) and at the LLaDA-8B
layout (multi-head attention, other tile widths), prefix 1024: one verify
forward of all 8 x 32 rows, every layer fed the GPU's own input residual stream
against the oracle's "fp8" mode layer (fixed rel-L2), and the oracle's FP8 LM
head + softmax on the GPU's own final rows (confidences within 1e-3, candidate
tokens equal at margins >= 1e-3, rows with an E4M3 tie in the final normed
values excused: either code is the rule applied). The block's tokens have no
E4M3 tie in their first normed rows; the prefix K/V are the GPU's own, read
back for the oracle."""
import types

import numpy as np
import pytest
import torch

import synth
from gpu_util import check_forward, log
from oracle import KVCache, OracleModel
from oracle.fp8 import E4M3_MAX, e4m3_round
from oracle.model import rms_norm

pytestmark = pytest.mark.gpu

L = 32


class _Layers:
    def __init__(self, w):
        self.w = w

    def __len__(self):
        return len(self.w["layers"])

    def __getitem__(self, i):
        return {k: v.float().cpu() for k, v in self.w["layers"][i].items()}


def _tie_free(rows, n, rng, eps):
    """n indices of rows (normed, unit weights) with no value at an E4M3 tie."""
    out = []
    for t in rng.permutation(len(rows)):
        h = rms_norm(rows[t][None], np.ones(rows.shape[1]), eps)[0]
        v = np.abs(h) * (E4M3_MAX / np.max(np.abs(h)))
        if np.array_equal(e4m3_round(v * (1 - 1e-6)), e4m3_round(v * (1 + 1e-6))):
            out.append(t)
            if len(out) == n:
                return np.array(out)
    raise AssertionError("not enough tie-free tokens")


@pytest.mark.parametrize("cfgname,P,K", [("dream7b_spread", 512, 7), ("dream7b_spread", 2048, 15),
                                         ("llada8b_spread", 1024, 7)])
def test_fp8_full_depth_all_rows(cfgname, P, K):
    import paper_2512_16229_amd as lp
    cfg = synth.config(cfgname)
    log(f"full shape {cfg['name']} fp8: prefix {P}, k {K}")
    w = synth.model_weights(cfg, device="cuda", dtype=torch.bfloat16)
    model = lp.Model(cfg, w, precision="fp8")
    kv = lp.KV(model, P + L, K + 1, L)
    dec = lp.Decoder(model, kv, L, K, 0.9)
    assert dec.prefill(synth.prompt(cfg, P, device="cuda")) == P
    rng = np.random.default_rng(12)
    cand = rng.choice(cfg["vocab"] - 1, 4096, replace=False)
    emb = w["embed"][torch.tensor(cand, device="cuda")].float().cpu().numpy().astype(np.float64)
    bt = cand[_tie_free(emb, (K + 1) * L, rng, cfg["rms_eps"])].reshape(K + 1, L)
    host = {"embed": w["embed"].float().cpu(), "layers": _Layers(w),
            "final_norm": w["final_norm"].float().cpu(), "lm_head": w["lm_head"].float().cpu()}
    cache = KVCache(cfg, P + L)
    for layer in range(cfg["layers"]):
        kg, vg = kv.read(layer, 0, P)
        cache.k[layer, :, :P] = kg.float().cpu().numpy()
        cache.v[layer, :, :P] = vg.float().cpu().numpy()
    s = types.SimpleNamespace(lp=lp, cfg=cfg, model=model, kv=kv, P=P, cache_f=cache,
                              faith=None)
    log("  quantising the oracle's FP8 LM head")
    s.faith = OracleModel(cfg, host, "fp8", keep_layers=1, bf16_weights=True)
    nb = K + 1
    conf_g = torch.empty(nb * L, dtype=torch.float32, device="cuda")
    pred_g = torch.empty(nb * L, dtype=torch.int32, device="cuda")
    lp.lopa_verify_forward(model, kv, P, torch.tensor(bt, dtype=torch.int32, device="cuda").reshape(-1),
                           nb, L, conf_g, pred_g)
    torch.cuda.synchronize()
    conf_g = conf_g.view(nb, L).cpu().numpy().astype(np.float64)
    pred_g = pred_g.view(nb, L).cpu().numpy()
    log(f"  conf {conf_g.min():.3f}..{conf_g.max():.3f}")
    # the first, a middle and the last layer fed the GPU's own input (the FP8
    # oracle quantises a layer's 233 M weights in tens of seconds)
    check_forward(s, bt, conf_g, pred_g, layers=[0, cfg["layers"] // 2, cfg["layers"] - 1],
                  label=f"{cfgname} fp8 verify forward")
