"""GPU parity of the batched verify forward (Alg. 1 step 3, Sec. 3.1, 3.3, 3.4)
against the oracle: confidences within 2e-2 of the float64 oracle, candidate
tokens equal to the bf16-faithful oracle except at near-ties (top-2
probability gap < 1e-3), prefix cache and branch staging equal to the oracle's
bf16 values up to rounding, and the batch properties (identical branches give
identical bits, permuted branches give permuted bits, repeat runs agree)."""
import numpy as np
import pytest
import torch

from gpu_util import Setup, conf_tolerance, faithful_bound, log, near_tie, vocab_margin

pytestmark = pytest.mark.gpu

# (config, P, L, k): 64 / 256 / 512 / 48 / 128 rows; ragged prefixes; two head dims
CASES = [("tiny", 64, 16, 3), ("small", 100, 32, 7), ("small", 37, 32, 15),
         ("small128", 40, 16, 2), ("small128", 0, 32, 3),
         # ragged and extreme block shapes: a 7-row block (partial key tile and
         # partial 16-row query block), 48 rows (three query blocks), the
         # 64-row maximum with head_dim 128, and the degenerate one-row block
         # with no prefix and no lookahead
         ("tiny", 23, 7, 2), ("small", 50, 48, 3), ("small128", 64, 64, 1), ("tiny", 0, 1, 0)]


def _kv_close(gpu, ref, what):
    g = gpu.float().cpu().numpy()
    scale = max(1.0, float(np.max(np.abs(ref))))
    err = np.abs(g - ref)
    assert err.max() <= 0.05 * scale, f"{what}: max err {err.max()} scale {scale}"
    assert err.mean() <= 2e-3 * scale, f"{what}: mean err {err.mean()}"


@pytest.mark.parametrize("cfgname,P,L,k", CASES)
def test_verify_forward_parity(cfgname, P, L, k):
    log(f"verify_forward parity {cfgname} P={P} L={L} k={k}")
    s = Setup(cfgname, P, L, k)
    s.gpu_prefill()
    # prefix cache after the GPU's own block-causal prefill
    for layer in range(s.cfg["layers"]):
        if P:
            kg, vg = s.kv.read(layer, 0, P)
            _kv_close(kg, s.cache_f.k[layer, :, :P], f"cache K layer {layer}")
            _kv_close(vg, s.cache_f.v[layer, :, :P], f"cache V layer {layer}")
    rng = np.random.default_rng(P + L + k)
    mask = s.cfg["mask_id"]
    nb = k + 1
    bt = np.where(rng.random((nb, L)) < 0.7, mask, rng.integers(0, s.cfg["vocab"] - 1, (nb, L)))
    bt[0] = mask
    # end to end (the GPU's own prefix cache): confidences
    conf, pred = s.gpu_forward(bt)
    rp = s.pure.forward_block(bt, P, s.cache_p)
    rf = s.faith.forward_block(bt, P, s.cache_f, keep_hidden=True)
    e_pure = np.max(np.abs(conf - rp["conf"]))
    e_bf16 = np.max(np.abs(rf["conf"] - rp["conf"]))   # the bf16 arithmetic itself, no GPU
    assert e_pure < conf_tolerance(e_bf16)
    # teacher-forced prefix (the oracle's cache): confidences and candidate tokens
    s.load_oracle_cache()
    conf, pred = s.gpu_forward(bt)
    marg = vocab_margin(rf["logits"], mask)
    e_faith = np.max(np.abs(conf - rf["conf"]))
    decided = marg >= near_tie(e_faith)
    log(f"  max|dconf| gpu-pure={e_pure:.2e} gpu-faithful={e_faith:.2e} faithful-pure={e_bf16:.2e} "
        f"near-ties={int((~decided).sum())}/{decided.size}")
    assert e_faith < faithful_bound(e_bf16)
    assert decided.mean() > 0.8
    assert np.array_equal(pred[decided], rf["pred"][decided]), \
        f"{int((pred[decided] != rf['pred'][decided]).sum())} decided tokens differ"
    assert not np.any(pred == mask)
    for j in (0, nb - 1):
        for layer in range(s.cfg["layers"]):
            ks, vs = s.kv.read_staging(j, layer, L)
            _kv_close(ks, rf["k"][j, layer], f"staging K b{j} l{layer}")
            _kv_close(vs, rf["v"][j, layer], f"staging V b{j} l{layer}")


@pytest.mark.parametrize("cfgname,P,L,k", [("tiny", 64, 16, 3), ("small", 100, 32, 7),
                                           ("small128", 40, 16, 1)])
def test_hidden_states_per_layer(cfgname, P, L, k):
    """Residual stream after every layer within rel-L2 1e-2 of the bf16-faithful oracle."""
    log(f"hidden states {cfgname} P={P} L={L} k={k}")
    s = Setup(cfgname, P, L, k)
    s.gpu_prefill()
    mask, nb = s.cfg["mask_id"], k + 1
    rng = np.random.default_rng(5)
    bt = np.where(rng.random((nb, L)) < 0.7, mask, rng.integers(0, s.cfg["vocab"] - 1, (nb, L)))
    btd = torch.tensor(bt, dtype=torch.int32, device="cuda").reshape(-1)
    for nl in range(s.cfg["layers"] + 1):
        x = torch.empty(nb * L * s.cfg["hidden"], dtype=torch.float32, device="cuda")
        s.lp.lopa_debug_hidden(s.model, s.kv, P, btd, nb, L, nl, x)
        torch.cuda.synchronize()
        g = x.view(nb, L, -1).cpu().numpy().astype(np.float64)
        r = s.faith.forward_block(bt, P, s.cache_f, n_layers=nl)["x"]
        rel = np.linalg.norm(g - r) / np.linalg.norm(r)
        log(f"  after {nl} layers: rel-L2 {rel:.2e}")
        assert rel < 1e-2
        if nl == 0:
            assert np.array_equal(g, r)          # embedding gather is exact


@pytest.mark.parametrize("cfgname,P,L,k", [("tiny", 64, 16, 3), ("small", 100, 32, 7),
                                           ("tiny", 23, 7, 2), ("small", 50, 48, 3)])
def test_batch_invariance_and_determinism(cfgname, P, L, k):
    log(f"batch invariance {cfgname} P={P} L={L} k={k}")
    s = Setup(cfgname, P, L, k)
    s.gpu_prefill()
    mask = s.cfg["mask_id"]
    nb = k + 1
    rng = np.random.default_rng(7)
    bt = np.where(rng.random((nb, L)) < 0.7, mask, rng.integers(0, s.cfg["vocab"] - 1, (nb, L)))
    c1, p1 = s.gpu_forward(bt)
    c2, p2 = s.gpu_forward(bt)
    assert np.array_equal(c1, c2) and np.array_equal(p1, p2)           # repeat: same bits
    dup = np.stack([bt[1]] * nb)
    cd, pd = s.gpu_forward(dup)
    assert all(np.array_equal(cd[0], cd[j]) for j in range(nb))        # identical rows: same bits
    perm = rng.permutation(nb)
    cp, pp = s.gpu_forward(bt[perm])
    assert np.array_equal(cp, c1[perm]) and np.array_equal(pp, p1[perm])
    # a branch alone gives the same bits as inside the batch of the same size
    one = np.stack([bt[2]] + [bt[2]] * (nb - 1))
    co, po = s.gpu_forward(one)
    assert np.array_equal(co[0], c1[2]) and np.array_equal(po[0], p1[2])
