"""GPU parity of the integer steps: branch construction (Eq. 1 + top-k), branch
scoring / selection (Eq. 2) and the winner's K/V commit, through the C ABI,
against the oracle on the same seeded inputs. Integer outputs bit-exact."""
import math

import numpy as np
import pytest
import torch

from gpu_util import f32, log
from oracle import lopa

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lp():
    import paper_2512_16229_amd as lp
    assert torch.cuda.is_available()
    return lp


def _dev(a, dtype):
    return torch.tensor(np.asarray(a), dtype=dtype, device="cuda").contiguous()


def _cases():
    rng = np.random.default_rng(1234)
    out = []
    for L in (1, 5, 16, 32, 33, 64, 65, 96, 128, 200, 256):
        for k in (0, 1, 3, 7, 15):
            for tau in (0.3, 0.9, 0.99):
                for style in ("cont", "ties"):
                    out.append((L, k, tau, style, int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("L,k,tau,style,seed", _cases())
def test_build_branches_matches_oracle(lp, L, k, tau, style, seed):
    log(f"build_branches L={L} k={k} tau={tau} {style} seed={seed}")
    rng = np.random.default_rng(seed)
    mask = 1000
    tokens = np.where(rng.random(L) < 0.75, mask, rng.integers(0, 1000, L)).astype(np.int32)
    if not (tokens == mask).any():
        tokens[rng.integers(L)] = mask
    conf = rng.random(L).astype(np.float32)
    if style == "ties":
        conf = (np.round(conf * 4) / 4).astype(np.float32)   # many exact ties, some == tau
    pred = rng.integers(0, 1000, L).astype(np.int32)
    nb = k + 1
    bt = torch.empty(nb * L, dtype=torch.int32, device="cuda")
    fp = torch.empty(nb, dtype=torch.int32, device="cuda")
    va = torch.empty(nb, dtype=torch.uint8, device="cuda")
    nv = torch.empty(1, dtype=torch.int32, device="cuda")
    lp.lopa_build_branches(_dev(tokens, torch.int32), _dev(conf, torch.float32),
                           _dev(pred, torch.int32), L, mask, tau, k, bt, fp, va, nv)
    torch.cuda.synchronize()
    rbt, rfp, rva, rnv = lopa.build_branches(tokens, conf.astype(np.float64), pred, mask, f32(tau), k)
    assert np.array_equal(bt.view(nb, L).cpu().numpy(), rbt)
    assert np.array_equal(fp.cpu().numpy(), rfp)
    assert np.array_equal(va.cpu().numpy(), rva)
    assert int(nv.item()) == rnv


METRICS = [(0, 1, 1.0), (1, 1, 1.0), (1, 3, 1.0), (1, 8, 1.0), (2, 1, 0.1), (2, 1, 0.25),
           (2, 1, 1.0)]


@pytest.mark.parametrize("metric,window,eta", METRICS, ids=lambda v: str(v))
@pytest.mark.parametrize("nb,L,seed", [(1, 16, 0), (4, 16, 1), (8, 32, 2), (16, 32, 3),
                                       (3, 7, 4), (8, 64, 5), (33, 9, 6), (4, 65, 7),
                                       (8, 128, 8), (2, 200, 9), (8, 256, 10)])
def test_select_matches_oracle(lp, nb, L, seed, metric, window, eta):
    """Eq. 2 (metric 0) and the alternative branch confidences (1: window
    minimum, 2: lowest-segment mean) against the oracle."""
    log(f"select nb={nb} L={L} seed={seed} metric={metric} window={window} eta={eta}")
    eta = f32(eta)
    rng = np.random.default_rng(seed)
    mask = 77
    for trial in range(20):
        bt = np.where(rng.random((nb, L)) < 0.6, mask, rng.integers(0, 77, (nb, L))).astype(np.int32)
        if trial % 5 == 0:
            bt[rng.integers(nb)] = 3                       # a complete branch -> +inf
        conf = rng.random((nb, L)).astype(np.float32)
        pred = rng.integers(0, 77, (nb, L)).astype(np.int32)
        valid = (rng.random(nb) < 0.8).astype(np.uint8)
        valid[0] = 1
        if trial % 7 == 0:                                 # identical rows
            bt[:] = bt[0]
            conf[:] = conf[0]
        out = dict(scores=torch.empty(nb, dtype=torch.float32, device="cuda"),
                   winner=torch.empty(1, dtype=torch.int32, device="cuda"),
                   nt=torch.empty(L, dtype=torch.int32, device="cuda"),
                   nc=torch.empty(L, dtype=torch.float32, device="cuda"),
                   np_=torch.empty(L, dtype=torch.int32, device="cuda"),
                   nu=torch.empty(1, dtype=torch.int32, device="cuda"))
        args = (_dev(bt.ravel(), torch.int32), _dev(conf.ravel(), torch.float32),
                _dev(pred.ravel(), torch.int32), _dev(valid, torch.uint8), nb, L, mask)
        outs = (out["scores"], out["winner"], out["nt"], out["nc"], out["np_"], out["nu"])
        if metric == 0 and trial % 2 == 0:
            lp.lopa_branch_confidence_select(*args, *outs)
        else:
            lp.lopa_branch_confidence_select_metric(*args, metric, window, eta, *outs)
        torch.cuda.synchronize()
        rs, rw = lopa.select(bt, conf.astype(np.float64), valid, mask, metric, window, eta)
        gs = out["scores"].cpu().numpy().astype(np.float64)
        fin = np.isfinite(rs)
        assert np.array_equal(np.isinf(gs), ~fin) and np.array_equal(np.sign(gs[~fin]), np.sign(rs[~fin]))
        assert np.max(np.abs(gs[fin] - rs[fin]), initial=0) < 1e-6
        w = int(out["winner"].item())
        s = np.sort(rs[np.isfinite(rs)])[::-1]
        tie = s.size > 1 and (s[0] - s[1]) < 1e-6 and not np.isposinf(rs).any()
        if not tie:
            assert np.array_equal(bt[w], bt[rw]) and w == rw
        if trial % 7 == 0:
            assert len(set(gs[valid == 1].tolist())) == 1 and w == 0   # identical rows: same bits
        assert np.array_equal(out["nt"].cpu().numpy(), bt[w])
        assert np.array_equal(out["nc"].cpu().numpy(), conf[w])
        assert np.array_equal(out["np_"].cpu().numpy(), pred[w])
        assert int(out["nu"].item()) == int((bt[w] == mask).sum())


def test_commit_copies_only_the_winner(lp):
    from gpu_util import Setup
    log("commit tiny P=32 L=16 k=3")
    s = Setup("tiny", 32, 16, 3)
    s.gpu_prefill()
    rng = np.random.default_rng(0)
    bt = np.where(rng.random((4, 16)) < 0.7, s.cfg["mask_id"], rng.integers(0, 1000, (4, 16)))
    s.gpu_forward(bt)
    off = torch.empty(1, dtype=torch.int32, device="cuda")
    for w in (2, 0, 3):
        s.lp.lopa_commit_kv(s.kv, torch.tensor([w], dtype=torch.int32, device="cuda"), 32, 16, off)
        torch.cuda.synchronize()
        assert int(off.item()) == 32
        for layer in range(s.cfg["layers"]):
            k, v = s.kv.read(layer, 32, 16)
            ks, vs = s.kv.read_staging(w, layer, 16)
            assert torch.equal(k, ks) and torch.equal(v, vs)
    before = [s.kv.read(l, 0, 48) for l in range(s.cfg["layers"])]
    for bad in (-1, 4, 100):
        s.lp.lopa_commit_kv(s.kv, torch.tensor([bad], dtype=torch.int32, device="cuda"), 32, 16, off)
        torch.cuda.synchronize()
        assert int(off.item()) == -1
    after = [s.kv.read(l, 0, 48) for l in range(s.cfg["layers"])]
    for (k0, v0), (k1, v1) in zip(before, after):
        assert torch.equal(k0, k1) and torch.equal(v0, v1)
    # capacity and mismatch errors are reported, not launched
    with pytest.raises(s.lp.LopaError):
        s.lp.lopa_commit_kv(s.kv, torch.zeros(1, dtype=torch.int32, device="cuda"), 31, 16, off)
    with pytest.raises(s.lp.LopaError):
        s.lp.lopa_verify_forward(s.model, s.kv, 60, torch.zeros(16, dtype=torch.int32, device="cuda"),
                                 1, 16, torch.empty(16, device="cuda"),
                                 torch.empty(16, dtype=torch.int32, device="cuda"))
