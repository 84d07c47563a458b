"""lopa_verify_forward_noalloc (working memory in the library's static device
array) against lopa_verify_forward (working memory of the KV handle) through
the C ABI: the same kernels on the same inputs give the same bits, for two
calls in a row with the second one smaller (the array keeps the first call's
contents), and a shape beyond the array's size is refused before anything
runs."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import log, to_dev_bf16

pytestmark = pytest.mark.gpu


def _run(lp, fn, model, kv, P, bt):
    nb, L = bt.shape
    btd = torch.tensor(bt, dtype=torch.int32, device="cuda").reshape(-1)
    conf = torch.full((nb * L,), float("nan"), dtype=torch.float32, device="cuda")
    pred = torch.full((nb * L,), -7, dtype=torch.int32, device="cuda")
    fn(model, kv, P, btd, nb, L, conf, pred)
    torch.cuda.synchronize()
    stag = [kv.read_staging(j, layer, L) for j in range(nb) for layer in (0, model.cfg["layers"] - 1)]
    return conf.cpu().numpy(), pred.cpu().numpy(), stag


@pytest.mark.parametrize("cfgname,precision", [("tiny", "bf16"), ("small128", "bf16"),
                                               ("small", "fp8")])
def test_noalloc_matches_the_allocating_entry(cfgname, precision):
    import paper_2512_16229_amd as lp
    cfg = synth.config(cfgname)
    model = lp.Model(cfg, to_dev_bf16(synth.model_weights(cfg)), precision=precision)
    P = 40
    kv = lp.KV(model, P + 32, 8, 32)
    dec = lp.Decoder(model, kv, 32, 7, 0.9)
    assert dec.prefill(synth.prompt(cfg, P)) == P
    rng = np.random.default_rng(4)
    mask = cfg["mask_id"]
    # two calls in a row, the second with fewer branches and a shorter block
    for nb, L in ((8, 32), (3, 7)):
        log(f"noalloc {cfgname} {precision}: {nb} branches x {L} rows")
        bt = np.where(rng.random((nb, L)) < 0.6, mask, rng.integers(0, cfg["vocab"] - 1, (nb, L)))
        c1, p1, s1 = _run(lp, lp.lopa_verify_forward_noalloc, model, kv, P, bt)
        c0, p0, s0 = _run(lp, lp.lopa_verify_forward, model, kv, P, bt)
        assert np.array_equal(c0, c1) and np.array_equal(p0, p1)
        for (k0, v0), (k1, v1) in zip(s0, s1):
            assert torch.equal(k0, k1) and torch.equal(v0, v1)
        # and the allocating entry again after the static one (nothing shared)
        c2, p2, _ = _run(lp, lp.lopa_verify_forward, model, kv, P, bt)
        assert np.array_equal(c0, c2) and np.array_equal(p0, p2)


def test_noalloc_refuses_a_shape_beyond_its_array():
    """A one-layer model whose gate/up operand alone (512 rows x 65536 columns
    of bf16, 64 MiB) exceeds the array: LOPA_ESHAPE, nothing enqueued; 64 rows
    of the same model fit."""
    import paper_2512_16229_amd as lp
    from paper_2512_16229_amd._abi import LopaError
    cfg = synth.config("tiny", layers=1, ffn=65536)
    model = lp.Model(cfg, to_dev_bf16(synth.model_weights(cfg)))
    kv = lp.KV(model, 64, 16, 32)
    bt = np.full((16, 32), cfg["mask_id"])
    with pytest.raises(LopaError) as e:
        _run(lp, lp.lopa_verify_forward_noalloc, model, kv, 0, bt)
    assert e.value.status == -2 and "working memory" in str(e.value)
    c1, p1, _ = _run(lp, lp.lopa_verify_forward_noalloc, model, kv, 0, bt[:2])
    c0, p0, _ = _run(lp, lp.lopa_verify_forward, model, kv, 0, bt[:2])
    assert np.array_equal(c0, c1) and np.array_equal(p0, p1)
