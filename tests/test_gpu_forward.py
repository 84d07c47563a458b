"""GPU parity of the batched verify forward (Alg. 1 step 3, Sec. 3.1, 3.3, 3.4)
against the oracle, with the fixed tolerances of gpu_util (check_forward):
confidences within 2e-2 of the float64 oracle on the same inputs; every layer,
fed the GPU's own input, within a fixed rel-L2 of the oracle layer; confidences
and candidate tokens of the oracle's LM head on the GPU's own final rows equal
except at near-ties (top-2 probability gap < 1e-3); prefix cache and branch
staging equal to the oracle's bf16 values up to rounding; and the batch
properties (identical branches give identical bits, permuted branches give
permuted bits, repeat runs agree)."""
import numpy as np
import pytest
import torch

from gpu_util import Setup, check_forward, gpu_residual, log, rel_l2

pytestmark = pytest.mark.gpu

# (config, P, L, k): 64 / 256 / 512 / 48 / 128 rows; ragged prefixes; two head dims; four widths
CASES = [("tiny", 64, 16, 3), ("small", 100, 32, 7), ("small", 37, 32, 15),
         ("small128", 40, 16, 2), ("small128", 0, 32, 3),
         # ragged and extreme block shapes: a 7-row block (partial key tile and
         # partial 16-row query block), 48 rows (three query blocks), the
         # 64-row maximum with head_dim 128, and the degenerate one-row block
         # with no prefix and no lookahead
         ("tiny", 23, 7, 2), ("small", 50, 48, 3), ("small128", 64, 64, 1), ("tiny", 0, 1, 0),
         # other widths (row kernels of 512 and 1024 x 2 threads' groups, other plans)
         ("wide1536", 64, 32, 3), ("wide6144", 40, 16, 3)]


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
    # teacher-forced prefix (the faithful oracle's cache rows)
    s.load_oracle_cache()
    conf, pred = s.gpu_forward(bt)
    st = check_forward(s, bt, conf, pred, label=f"{cfgname} P={P} L={L} k={k}")
    rf = st["faith"]
    for j in (0, nb - 1):
        for layer in range(s.cfg["layers"]):
            ks, vs = s.kv.read_staging(j, layer, L)
            _kv_close(ks, rf["k"][j, layer], f"staging K b{j} l{layer}")
            _kv_close(vs, rf["v"][j, layer], f"staging V b{j} l{layer}")


# long prefixes (many key tiles per wavefront, ragged last tile) with 4 to 16
# branches, and short ones down to a single prefix key
LONG = [("tiny", 512, 16, 3), ("small", 600, 32, 15), ("small128", 300, 32, 15),
        ("tiny", 37, 16, 3), ("small128", 1, 8, 2), ("small", 100, 48, 3),
        # past 24 key tiles: the grouped form (key splits, one K / V tile per
        # KV head for all its query heads)
        ("small", 1000, 32, 7), ("small128", 900, 16, 3), ("tiny", 1200, 16, 1)]


@pytest.mark.parametrize("cfgname,P,L,k", LONG)
def test_long_prefix_attention(cfgname, P, L, k):
    """Prefix lengths from one key to many tiles per wavefront against the
    oracle (every row sees the whole committed prefix, Sec. 3.3)."""
    log(f"prefix attention {cfgname} P={P} L={L} k={k}")
    s = Setup(cfgname, P, L, k)
    s.gpu_prefill()
    s.load_oracle_cache()
    nb, mask = k + 1, s.cfg["mask_id"]
    rng = np.random.default_rng(P + 3 * L + k)
    bt = np.where(rng.random((nb, L)) < 0.7, mask, rng.integers(0, s.cfg["vocab"] - 1, (nb, L)))
    bt[0] = mask
    conf, pred = s.gpu_forward(bt)
    check_forward(s, bt, conf, pred, label=f"prefix {P}")


@pytest.mark.parametrize("cfgname,P,L,k", [("tiny", 64, 16, 3), ("small", 100, 32, 7),
                                           ("small128", 40, 16, 1)])
def test_hidden_states_per_layer(cfgname, P, L, k):
    """The residual stream after every layer of the GPU's own forward (its own
    prefill too) against the faithful oracle's end to end: rel-L2 within 1e-2
    at every depth, the embedding gather exact."""
    log(f"hidden states {cfgname} P={P} L={L} k={k}")
    s = Setup(cfgname, P, L, k)
    s.gpu_prefill()
    mask, nb = s.cfg["mask_id"], k + 1
    rng = np.random.default_rng(5)
    bt = np.where(rng.random((nb, L)) < 0.7, mask, rng.integers(0, s.cfg["vocab"] - 1, (nb, L)))
    for nl in range(s.cfg["layers"] + 1):
        g = gpu_residual(s, bt, nl)
        r = s.faith.forward_block(bt, P, s.cache_f, n_layers=nl)["x"]
        rel = rel_l2(g, r)
        log(f"  after {nl} layers: rel-L2 {rel:.2e}")
        assert rel < 1e-2
        if nl == 0:
            assert np.array_equal(g, r)          # embedding gather is exact


@pytest.mark.parametrize("cfgname,P,L,k", [("tiny", 64, 16, 3), ("small", 100, 32, 7),
                                           ("tiny", 23, 7, 2), ("small", 50, 48, 3),
                                           ("tiny", 300, 7, 15), ("small", 400, 24, 7)])
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


# (config, P, L, k, sub-block): the block-causal mask inside the block (Sec.
# 3.4, the Ascend system's mask); 16-row sub-blocks make a 32-key tile partly
# visible to a row block
CAUSAL = [("small", 100, 64, 3, 32), ("small", 300, 64, 3, 32), ("tiny", 40, 48, 2, 16),
          ("tiny", 272, 48, 5, 16), ("small128", 64, 64, 1, 16),
          ("small", 900, 32, 3, 16)]  # the grouped form with the mask


@pytest.mark.parametrize("cfgname,P,L,k,cblk", CAUSAL)
def test_block_causal_forward(cfgname, P, L, k, cblk):
    log(f"block-causal forward {cfgname} P={P} L={L} k={k} sub-block {cblk}")
    s = Setup(cfgname, P, L, k)
    s.gpu_prefill()
    s.load_oracle_cache()
    nb, mask = k + 1, s.cfg["mask_id"]
    s.kv.set_block_causal(cblk)
    rng = np.random.default_rng(P + L + cblk)
    bt = np.where(rng.random((nb, L)) < 0.6, mask, rng.integers(0, s.cfg["vocab"] - 1, (nb, L)))
    conf, pred = s.gpu_forward(bt)
    st = check_forward(s, bt, conf, pred, causal_blk=cblk, label=f"block-causal {cblk}")
    rf = st["faith"]
    # the mask matters: the unmasked oracle differs by more than the tolerance
    # somewhere in the first sub-block
    full = s.faith.forward_block(bt, P, s.cache_f)
    assert np.max(np.abs(full["conf"][:, :cblk] - rf["conf"][:, :cblk])) > 0
    # staged K / V of the last sub-block, and a block of one sub-block is unmasked
    for layer in range(s.cfg["layers"]):
        ks, vs = s.kv.read_staging(nb - 1, layer, L)
        _kv_close(ks, rf["k"][nb - 1, layer], f"staging K l{layer}")
        _kv_close(vs, rf["v"][nb - 1, layer], f"staging V l{layer}")
    s.kv.set_block_causal(0)
