"""GPU parity at the full model shapes of the measured workloads, in the launch
configuration bench.py times (every plan and kernel of the step at that size):
  * Dream-7B, prefix 512, k = 7 (8 branches x 32 rows: one 256-row tile);
  * Dream-7B, prefix 2048, k = 15 (16 branches x 32 rows: two row tiles);
  * LLaDA-8B (MHA, no biases), prefix 1024, k = 7.

The oracle cannot run 28-32 float64 layers at these sizes in seconds, so outputs
are sampled where it can compute them one by one:
  * the residual stream after the first layer for every row (one float64
    layer, the prefix K/V of that layer taken from the GPU's own cache);
  * Conf / candidate token of sampled rows from the GPU's final residual stream:
    final RMSNorm + the full-vocabulary LM head + softmax in float64 (Sec. 3.1).
The LM head is spread (N(0, 8/sqrt(H))) so that confidences are informative."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import conf_tolerance, faithful_bound, log, near_tie, vocab_margin
from oracle import KVCache, OracleModel
from oracle.model import bf16_round, confidence, rms_norm

pytestmark = pytest.mark.gpu

L = 32
CASES = [("dream7b_spread", 512, 7), ("dream7b_spread", 2048, 15), ("llada8b_spread", 1024, 7)]


@pytest.fixture(scope="module", params=CASES, ids=lambda c: f"{c[0]}-P{c[1]}-k{c[2]}")
def big(request):
    import paper_2512_16229_amd as lp
    name, P, K = request.param
    log(f"full shape {name}: prefix {P}, k {K}")
    cfg = synth.config(name)
    w = synth.model_weights(cfg, device="cuda", dtype=torch.bfloat16)
    model = lp.Model(cfg, w)
    kv = lp.KV(model, P + L, K + 1, L)
    dec = lp.Decoder(model, kv, L, K, 0.9)
    assert dec.prefill(synth.prompt(cfg, P, device="cuda")) == P
    rng = np.random.default_rng(11)
    mask = cfg["mask_id"]
    bt = np.where(rng.random((K + 1, L)) < 0.7, mask, rng.integers(0, cfg["vocab"] - 1, (K + 1, L)))
    bt[0] = mask
    torch.cuda.synchronize()
    yield dict(lp=lp, cfg=cfg, w=w, model=model, kv=kv, bt=bt, P=P)
    del dec, kv, model, w
    torch.cuda.empty_cache()


def _hidden(big, n_layers):
    lp, cfg, bt, P = big["lp"], big["cfg"], big["bt"], big["P"]
    nb = bt.shape[0]
    x = torch.empty(nb * L * cfg["hidden"], dtype=torch.float32, device="cuda")
    btd = torch.tensor(bt, dtype=torch.int32, device="cuda").reshape(-1)
    lp.lopa_debug_hidden(big["model"], big["kv"], P, btd, nb, L, n_layers, x)
    torch.cuda.synchronize()
    return x.view(nb, L, -1).cpu().numpy().astype(np.float64)


def test_first_layer_all_rows(big):
    cfg, w, bt, P = big["cfg"], big["w"], big["bt"], big["P"]
    log(f"  layer 0, {bt.size} rows, prefix {P}")
    g = _hidden(big, 1)
    cfg1 = dict(cfg, layers=1)
    host = {"embed": w["embed"].float().cpu(),
            "layers": [{k: v.float().cpu() for k, v in w["layers"][0].items()}],
            "final_norm": w["final_norm"].float().cpu(),
            "lm_head": w["lm_head"][:1].float().cpu()}        # not reached with n_layers=1
    faith = OracleModel(cfg1, host, "faithful")
    del host
    cache = KVCache(cfg1, P + L)
    kg, vg = big["kv"].read(0, 0, P)                          # the GPU's prefix, layer 0 (bf16)
    cache.k[0, :, :P] = kg.float().cpu().numpy()
    cache.v[0, :, :P] = vg.float().cpu().numpy()
    r = faith.forward_block(bt, P, cache, n_layers=1)["x"]
    rel = np.linalg.norm(g - r) / np.linalg.norm(r)
    log(f"  residual stream after layer 0: rel-L2 {rel:.2e}")
    assert rel < 1e-2


def test_lm_head_sampled_rows(big):
    lp, cfg, w, bt, P = big["lp"], big["cfg"], big["w"], big["bt"], big["P"]
    log("  LM head + Conf on sampled rows, full vocabulary")
    nb = bt.shape[0]
    conf_g = torch.empty(nb * L, dtype=torch.float32, device="cuda")
    pred_g = torch.empty(nb * L, dtype=torch.int32, device="cuda")
    btd = torch.tensor(bt, dtype=torch.int32, device="cuda").reshape(-1)
    lp.lopa_verify_forward(big["model"], big["kv"], P, btd, nb, L, conf_g, pred_g)
    torch.cuda.synchronize()
    conf_g = conf_g.cpu().numpy().astype(np.float64)
    pred_g = pred_g.cpu().numpy()
    x = _hidden(big, cfg["layers"]).reshape(nb * L, -1)
    rows = np.random.default_rng(3).choice(nb * L, 24, replace=False)
    lm = w["lm_head"].float().cpu().numpy().astype(np.float64)   # bf16 values
    fn = w["final_norm"].float().cpu().numpy().astype(np.float64)
    h = rms_norm(x[rows], fn, cfg["rms_eps"])
    lg_pure = h @ lm.T
    lg_faith = bf16_round(h) @ lm.T                              # the LM head's operand is bf16
    cp, _ = confidence(lg_pure, cfg["mask_id"])
    cf, pf = confidence(lg_faith, cfg["mask_id"])
    e_bf16 = np.max(np.abs(cf - cp))
    e = np.max(np.abs(conf_g[rows] - cf))
    log(f"  max|dconf| gpu-faithful {e:.2e}, gpu-pure {np.max(np.abs(conf_g[rows] - cp)):.2e}, "
        f"faithful-pure {e_bf16:.2e}; conf range {cf.min():.3f}..{cf.max():.3f}")
    assert e < faithful_bound(e_bf16)
    assert np.max(np.abs(conf_g[rows] - cp)) < conf_tolerance(e_bf16)
    decided = vocab_margin(lg_faith, cfg["mask_id"]) >= near_tie(e)
    assert decided.mean() > 0.8
    assert np.array_equal(pred_g[rows][decided], pf[decided])
