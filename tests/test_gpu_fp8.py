"""GPU parity of the FP8 MLP model mode (lopa_model_create_ex with
LOPA_PRECISION_FP8_MLP: gate / up / down in W8A8 E4M3) against the oracle's
FP8 mode, which quantises at the same points with the same rules.

Teacher-forced prefix (the oracle's cache rows), then: confidences within the
case's own tolerance (2e-2, or a few times the oracle's own sensitivity to
bf16-sized perturbations, which E4M3 rounding amplifies), candidate tokens
equal except at near-ties, the first layer to float32-rounding accuracy where
attention is exact (one key per row), and the batch properties (identical
branches give identical bits, permuted branches permuted bits)."""
import numpy as np
import pytest
import torch

from gpu_util import Setup, conf_tolerance, log, near_tie, vocab_margin

pytestmark = pytest.mark.gpu

# (config, P, L, k): two head dims, a ragged block, and the shared-prefix
# attention path (P = 300, 16 branches)
CASES = [("tiny", 64, 16, 3), ("small", 100, 32, 7), ("small128", 40, 16, 2), ("tiny", 23, 7, 2),
         ("small", 300, 32, 15)]


def _tokens(s, nb, L, seed):
    rng = np.random.default_rng(seed)
    mask = s.cfg["mask_id"]
    bt = np.where(rng.random((nb, L)) < 0.7, mask, rng.integers(0, s.cfg["vocab"] - 1, (nb, L)))
    bt[0] = mask
    return bt


def _sensitivity(s, bt, P, base_conf, seed=0):
    """How far the oracle's own FP8 confidences move when the prefix K/V are
    perturbed by a quarter of a bf16 step (relative 2^-10, random sign): the
    E4M3 roundings turn such differences - the size of the GPU's rounding-order
    differences in the bf16 parts - into whole-code changes, and the synthetic
    LM heads amplify them. The GPU may differ from the oracle by a few times this."""
    rng = np.random.default_rng(seed)
    c2 = s.cache_f.copy()
    c2.k *= 1.0 + rng.choice([-1.0, 1.0], c2.k.shape) * 2.0 ** -10
    c2.v *= 1.0 + rng.choice([-1.0, 1.0], c2.v.shape) * 2.0 ** -10
    return float(np.max(np.abs(s.faith.forward_block(bt, P, c2)["conf"] - base_conf)))


@pytest.mark.parametrize("cfgname,P,L,k", CASES)
def test_fp8_forward_parity(cfgname, P, L, k):
    log(f"fp8 forward {cfgname} P={P} L={L} k={k}")
    s = Setup(cfgname, P, L, k, precision="fp8_mlp")
    s.load_oracle_cache()
    nb, mask = k + 1, s.cfg["mask_id"]
    bt = _tokens(s, nb, L, P + L + k)
    conf, pred = s.gpu_forward(bt)
    rf = s.faith.forward_block(bt, P, s.cache_f, keep_hidden=True)
    e = np.max(np.abs(conf - rf["conf"]))
    sens = _sensitivity(s, bt, P, rf["conf"]) if P else 0.0
    decided = vocab_margin(rf["logits"], mask) >= near_tie(e)
    log(f"  max|dconf| gpu-oracle(fp8)={e:.2e}, oracle sensitivity {sens:.2e}, "
        f"decided {decided.mean():.2f}")
    assert e < max(conf_tolerance(0.0), 4.0 * sens)
    if sens < conf_tolerance(0.0):  # otherwise the near-tie band may cover most rows
        assert decided.mean() > 0.5
    assert np.array_equal(pred[decided], rf["pred"][decided])
    assert not np.any(pred == mask)


@pytest.mark.parametrize("cfgname", ["tiny", "small", "small128"])
def test_fp8_first_layer_single_key(cfgname):
    """No prefix and one-row blocks: every row attends to itself only, so the
    bf16 parts agree with the oracle to float32 rounding and the first layer's
    residual stream isolates the FP8 MLP (weight repack, per-row scales of the
    RMSNorm output, FP8 GEMMs, SwiGLU, requantisation, down projection). The
    bound covers the rare whole-code changes that bf16 rounding-order
    differences of the SwiGLU output cause in its requantisation; a wrong
    layout or scale would be off by order one."""
    s = Setup(cfgname, 0, 1, 7, precision="fp8_mlp")
    nb = 8
    bt = np.random.default_rng(1).integers(0, s.cfg["vocab"] - 1, (nb, 1))
    btd = torch.tensor(bt, dtype=torch.int32, device="cuda").reshape(-1)
    x = torch.empty(nb * s.cfg["hidden"], dtype=torch.float32, device="cuda")
    s.lp.lopa_debug_hidden(s.model, s.kv, 0, btd, nb, 1, 1, x)
    torch.cuda.synchronize()
    g = x.view(nb, 1, -1).cpu().numpy().astype(np.float64)
    r = s.faith.forward_block(bt, 0, s.cache_f, n_layers=1)["x"]
    rel = np.linalg.norm(g - r) / np.linalg.norm(r)
    log(f"fp8 first layer, single key, {cfgname}: rel-L2 {rel:.2e}")
    assert rel < 2e-3


@pytest.mark.parametrize("cfgname,P,L,k", [("tiny", 64, 16, 3), ("small", 50, 48, 3)])
def test_fp8_batch_invariance(cfgname, P, L, k):
    """Per-row activation scales keep rows independent: identical branches give
    identical bits, permuted branches permuted bits, repeats the same bits."""
    s = Setup(cfgname, P, L, k, precision="fp8_mlp")
    s.load_oracle_cache()
    nb = k + 1
    bt = _tokens(s, nb, L, 9)
    c1, p1 = s.gpu_forward(bt)
    c2, p2 = s.gpu_forward(bt)
    assert np.array_equal(c1, c2) and np.array_equal(p1, p2)
    cd, _ = s.gpu_forward(np.stack([bt[1]] * nb))
    assert all(np.array_equal(cd[0], cd[j]) for j in range(nb))
    perm = np.random.default_rng(3).permutation(nb)
    cp, pp = s.gpu_forward(bt[perm])
    assert np.array_equal(cp, c1[perm]) and np.array_equal(pp, p1[perm])


def test_fp8_decode_block():
    """The FP8 model through the decode loop: the block fills within L
    iterations and nothing stays masked (the oracle's FP8 trajectory is logged
    beside it)."""
    from oracle import lopa
    s = Setup("tiny", 64, 16, 3, precision="fp8_mlp")
    dec = s.gpu_prefill()
    s.load_oracle_cache()
    iters = dec.decode_block(64)
    toks = dec.tokens.cpu().numpy()
    assert 1 <= iters <= 16 and not np.any(toks == s.cfg["mask_id"])
    otoks, oiters, _ = lopa.decode_block(s.faith, s.cache_f.copy(), 64, 16, 3, np.float32(0.9))
    log(f"  fp8 decode: {iters} iterations (oracle {oiters}), "
        f"{int(np.sum(toks == otoks))}/16 tokens equal")
