"""GPU parity of the FP8 model mode (LOPA_PRECISION_FP8: QKV, gate / up / down
and the LM head in W8A8 E4M3) at the full Dream-7B shape, prefix 512, k = 7, in
the launch configuration bench.py times for its FP8 step figure. As for the bf16
full-shape tests, outputs are sampled where the float64 oracle can compute them:
  * the residual stream after the first layer for every row (the oracle's "fp8"
    mode over one layer, the prefix K/V of that layer taken from the GPU's own
    cache), within a few times the oracle's own sensitivity to bf16-sized
    perturbations; the block's tokens have no E4M3 tie in their first normed
    rows, so one code sequence of the QKV operand is correct (a tie is decided
    either way by float32 roundings and moves its row by about a percent);
  * Conf / candidate token of sampled rows from the GPU's final residual stream:
    final RMSNorm, per-row E4M3 quantisation, the quantised full-vocabulary LM
    head, softmax (Sec. 3.1)."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import log, vocab_margin
from oracle import KVCache, OracleModel
from oracle.fp8 import E4M3_MAX, e4m3_round, quantize_rows
from oracle.model import confidence, rms_norm

pytestmark = pytest.mark.gpu

L, P, K = 32, 512, 7


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


@pytest.fixture(scope="module")
def big():
    import paper_2512_16229_amd as lp
    cfg = synth.config("dream7b_spread")
    log(f"full shape {cfg['name']} fp8: prefix {P}, k {K}")
    w = synth.model_weights(cfg, device="cuda", dtype=torch.bfloat16)
    model = lp.Model(cfg, w, precision="fp8")
    kv = lp.KV(model, P + L, K + 1, L)
    dec = lp.Decoder(model, kv, L, K, 0.9)
    assert dec.prefill(synth.prompt(cfg, P, device="cuda")) == P
    # candidate tokens: a random sample of the vocabulary, tie-free ones kept
    rng = np.random.default_rng(12)
    cand = rng.choice(cfg["vocab"] - 1, 2048, replace=False)
    emb = w["embed"][torch.tensor(cand, device="cuda")].float().cpu().numpy().astype(np.float64)
    bt = cand[_tie_free(emb, (K + 1) * L, rng, cfg["rms_eps"])].reshape(K + 1, L)
    torch.cuda.synchronize()
    yield dict(lp=lp, cfg=cfg, w=w, model=model, kv=kv, bt=bt)
    del dec, kv, model, w
    torch.cuda.empty_cache()


def _hidden(big, n_layers):
    lp, cfg, bt = big["lp"], big["cfg"], big["bt"]
    nb = bt.shape[0]
    x = torch.empty(nb * L * cfg["hidden"], dtype=torch.float32, device="cuda")
    btd = torch.tensor(bt, dtype=torch.int32, device="cuda").reshape(-1)
    lp.lopa_debug_hidden(big["model"], big["kv"], P, btd, nb, L, n_layers, x)
    torch.cuda.synchronize()
    return x.view(nb, L, -1).cpu().numpy().astype(np.float64)


def test_fp8_first_layer_all_rows(big):
    cfg, w, bt = big["cfg"], big["w"], big["bt"]
    g = _hidden(big, 1)
    cfg1 = dict(cfg, layers=1)
    host = {"embed": w["embed"].float().cpu(),
            "layers": [{k: v.float().cpu() for k, v in w["layers"][0].items()}],
            "final_norm": w["final_norm"].float().cpu(),
            "lm_head": w["lm_head"][:1].float().cpu()}        # not reached with n_layers=1
    orc = OracleModel(cfg1, host, "fp8")
    del host
    cache = KVCache(cfg1, P + L)
    kg, vg = big["kv"].read(0, 0, P)                          # the GPU's prefix, layer 0 (bf16)
    cache.k[0, :, :P] = kg.float().cpu().numpy()
    cache.v[0, :, :P] = vg.float().cpu().numpy()
    r = orc.forward_block(bt, P, cache, n_layers=1)["x"]
    rel = np.linalg.norm(g - r) / np.linalg.norm(r)
    # the oracle's own sensitivity: the prefix K/V moved by a quarter of a bf16
    # step (relative 2^-10, random sign). Bf16-sized differences upstream of
    # the MLP flip some E4M3 codes of its two quantised operands, and at this
    # width (3584 and 18944 values per row) many, so the first layer's output
    # moves by percents in both the oracle and the GPU.
    rng = np.random.default_rng(0)
    c2 = cache.copy()
    c2.k *= 1.0 + rng.choice([-1.0, 1.0], c2.k.shape) * 2.0 ** -10
    c2.v *= 1.0 + rng.choice([-1.0, 1.0], c2.v.shape) * 2.0 ** -10
    r2 = orc.forward_block(bt, P, c2, n_layers=1)["x"]
    sens = np.linalg.norm(r2 - r) / np.linalg.norm(r)
    log(f"  fp8 residual stream after layer 0: rel-L2 {rel:.2e}, oracle sensitivity {sens:.2e}")
    assert rel < max(1e-2, 3.0 * sens)


def test_fp8_lm_head_sampled_rows(big):
    lp, cfg, w, bt = big["lp"], big["cfg"], big["w"], big["bt"]
    nb = bt.shape[0]
    conf_g = torch.empty(nb * L, dtype=torch.float32, device="cuda")
    pred_g = torch.empty(nb * L, dtype=torch.int32, device="cuda")
    btd = torch.tensor(bt, dtype=torch.int32, device="cuda").reshape(-1)
    lp.lopa_verify_forward(big["model"], big["kv"], P, btd, nb, L, conf_g, pred_g)
    torch.cuda.synchronize()
    conf_g = conf_g.cpu().numpy().astype(np.float64)
    pred_g = pred_g.cpu().numpy()
    x = _hidden(big, cfg["layers"]).reshape(nb * L, -1)
    rows = np.random.default_rng(3).choice(nb * L, 48, replace=False)
    fn = w["final_norm"].float().cpu().numpy().astype(np.float64)
    hf = rms_norm(x[rows], fn, cfg["rms_eps"])
    # the LM head's per-row quantisation, in vocabulary chunks
    lm = w["lm_head"].float().cpu().numpy()
    qx, sx = quantize_rows(hf)
    logits = np.empty((len(rows), cfg["vocab"]))
    for c0 in range(0, cfg["vocab"], 16384):
        qw, sw = quantize_rows(lm[c0:c0 + 16384])
        logits[:, c0:c0 + 16384] = (qx @ qw.T) * sx[:, None] * sw
    del lm
    rc, rp = confidence(logits, cfg["mask_id"])
    v = np.abs(hf) * (E4M3_MAX / np.max(np.abs(hf), axis=-1, keepdims=True))
    # (3584 values per row: a margin of a few float32 steps keeps most rows)
    clear = np.all(e4m3_round(v * (1 - 2e-6)) == e4m3_round(v * (1 + 2e-6)), axis=-1)
    e = np.max(np.abs(conf_g[rows] - rc)[clear])
    decided = (vocab_margin(logits, cfg["mask_id"]) >= 1e-3) & clear
    log(f"  fp8 LM head on sampled rows: max|dconf| {e:.2e}, rows without ties {clear.mean():.2f}, "
        f"decided {decided.mean():.2f}; conf range {rc.min():.3f}..{rc.max():.3f}")
    assert clear.mean() > 0.5 and e < 5e-4
    assert decided.mean() > 0.4 and np.array_equal(pred_g[rows][decided], rp[decided])
