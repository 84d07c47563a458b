"""Pins of the oracle forward (oracle/model.py) against torch CPU library ops.

An independent float64 torch implementation written here (F.rms_norm,
F.scaled_dot_product_attention with an explicit mask, F.silu, RoPE as a
complex rotation) computes the full-sequence forward with a block-causal mask
and no cache. The oracle's cached block forward must agree with it, which pins
the attention pattern of Sec. 3.3 (full attention inside the active block, the
committed prefix visible, branches isolated) and the static cache + commit of
Sec. 3.4."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import KVCache, OracleModel, bf16_round, lopa
from oracle.model import apply_rope, rms_norm, rope_angles, silu


def _tiny(**over):
    cfg = synth.config("tiny", **over)
    return cfg, synth.model_weights(cfg)


# ------------------------------------------------------------------ pieces
def test_rms_norm_matches_torch():
    x = np.random.default_rng(0).normal(size=(7, 33))
    w = np.random.default_rng(1).normal(size=33)
    ref = F.rms_norm(torch.tensor(x), (33,), torch.tensor(w), eps=1e-6).numpy()
    assert np.allclose(rms_norm(x, w, 1e-6), ref, rtol=1e-13, atol=1e-14)


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    assert np.allclose(silu(x), F.silu(torch.tensor(x)).numpy(), rtol=1e-13, atol=1e-300)


def _rope_complex(x, pos, theta):
    d = x.shape[-1]
    ang = torch.outer(torch.tensor(pos, dtype=torch.float64),
                      theta ** (-torch.arange(0, d, 2, dtype=torch.float64) / d))
    z = torch.complex(x[..., : d // 2], x[..., d // 2:]) * torch.polar(torch.ones_like(ang), ang)
    return torch.cat([z.real, z.imag], dim=-1)


def test_rope_is_a_complex_rotation_and_relative():
    rng = np.random.default_rng(2)
    x = rng.normal(size=(3, 5, 64))
    pos = np.arange(40, 45)
    got = apply_rope(x, rope_angles(pos, 64, 1e4))
    ref = _rope_complex(torch.tensor(x), pos, 1e4).numpy()
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)
    # scores depend only on the position difference
    q, k = rng.normal(size=(1, 64)), rng.normal(size=(1, 64))
    for m, n, c in [(3, 9, 100), (0, 0, 7), (500, 2, 1000)]:
        a = apply_rope(q, rope_angles(np.array([m]), 64, 1e4)) @ apply_rope(k, rope_angles(np.array([n]), 64, 1e4)).T
        b = apply_rope(q, rope_angles(np.array([m + c]), 64, 1e4)) @ apply_rope(k, rope_angles(np.array([n + c]), 64, 1e4)).T
        assert abs(a - b) < 1e-10


def test_bf16_round_matches_torch():
    x = np.concatenate([np.random.default_rng(3).normal(0, 1, 10000),
                        [0.0, -0.0, 1e-40, 3.0e38, 1 + 2 ** -8, 1 + 3 * 2 ** -8]])
    ref = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(bf16_round(x), ref)


# --------------------------------------------------------- torch reference
def torch_full_forward(cfg, w, seq, allowed):
    """Full-sequence forward over `seq` (T tokens at positions 0..T-1) with the
    boolean attention mask allowed[i, j]; returns (logits [T, V], k, v per layer)."""
    d, Hq, Hkv = cfg["head_dim"], cfg["heads"], cfg["kv_heads"]
    T = len(seq)
    t = lambda a: a.to(torch.float64)
    x = t(w["embed"])[torch.tensor(seq)]
    am = torch.tensor(allowed)
    ks, vs = [], []
    for lw in w["layers"]:
        h = F.rms_norm(x, (cfg["hidden"],), t(lw["ln1"]), eps=cfg["rms_eps"])
        q, k, v = h @ t(lw["wq"]).T, h @ t(lw["wk"]).T, h @ t(lw["wv"]).T
        if cfg["qkv_bias"]:
            q, k, v = q + t(lw["bq"]), k + t(lw["bk"]), v + t(lw["bv"])
        q = q.view(T, Hq, d).transpose(0, 1)
        k = k.view(T, Hkv, d).transpose(0, 1)
        v = v.view(T, Hkv, d).transpose(0, 1)
        q = _rope_complex(q, np.arange(T), cfg["rope_theta"])
        k = _rope_complex(k, np.arange(T), cfg["rope_theta"])
        ks.append(k)
        vs.append(v)
        rep = Hq // Hkv
        o = F.scaled_dot_product_attention(q[None], k.repeat_interleave(rep, 0)[None],
                                           v.repeat_interleave(rep, 0)[None], attn_mask=am)[0]
        x = x + o.transpose(0, 1).reshape(T, Hq * d) @ t(lw["wo"]).T
        h2 = F.rms_norm(x, (cfg["hidden"],), t(lw["ln2"]), eps=cfg["rms_eps"])
        x = x + (F.silu(h2 @ t(lw["w_gate"]).T) * (h2 @ t(lw["w_up"]).T)) @ t(lw["w_down"]).T
    hf = F.rms_norm(x, (cfg["hidden"],), t(w["final_norm"]), eps=cfg["rms_eps"])
    return (hf @ t(w["lm_head"]).T).numpy(), ks, vs


def block_causal(T, L):
    b = np.arange(T) // L
    return b[:, None] >= b[None, :]


def _conf_pred(logits, mask_id):
    lg = logits.copy()
    lg[:, mask_id] = -np.inf
    p = np.exp(lg - lg.max(-1, keepdims=True))
    p /= p.sum(-1, keepdims=True)
    return p.max(-1), p.argmax(-1)


@pytest.mark.parametrize("cfgname,P,L", [("tiny", 48, 16), ("small128", 20, 8)])
def test_cached_block_forward_equals_full_sequence(cfgname, P, L):
    """Prefill (block-causal, committed block by block) + one block forward against the
    cache == full-sequence forward with a block-causal mask.  Ragged last prefill block
    in the second case (20 = 2*8 + 4)."""
    cfg = synth.config(cfgname)
    if cfgname == "small128":
        cfg["layers"] = 1
    w = synth.model_weights(cfg)
    m = OracleModel(cfg, w)
    prompt = synth.prompt(cfg, P).numpy()
    cache = KVCache(cfg, P + L)
    assert lopa.prefill(m, cache, prompt, L) == P
    rng = np.random.default_rng(4)
    blk = np.where(rng.random(L) < 0.6, cfg["mask_id"], rng.integers(0, cfg["vocab"] - 1, L))
    out = m.forward_block(blk[None], P, cache)
    seq = np.concatenate([prompt, blk])
    # prefill blocks have boundaries at multiples of L from 0; the active block starts at P
    bid = np.concatenate([np.arange(P) // L, np.full(L, (P + L - 1) // L + 1)])
    allowed = bid[:, None] >= bid[None, :]
    logits, ks, vs = torch_full_forward(cfg, w, seq, allowed)
    conf, pred = _conf_pred(logits[P:], cfg["mask_id"])
    assert np.allclose(out["conf"][0], conf, rtol=1e-9, atol=1e-12)
    assert np.array_equal(out["pred"][0], pred)
    for li in range(cfg["layers"]):
        assert np.allclose(cache.k[li, :, :P], ks[li][:, :P].numpy(), atol=1e-10)
        assert np.allclose(cache.v[li, :, :P], vs[li][:, :P].numpy(), atol=1e-10)
        assert np.allclose(out["k"][0, li], ks[li][:, P:].numpy(), atol=1e-10)
        assert np.allclose(out["v"][0, li], vs[li][:, P:].numpy(), atol=1e-10)


def test_branch_isolation_batched_equals_single():
    """Row block j of one batched forward == the forward of branch j alone (Alg. 1 step 3)."""
    cfg, w = _tiny()
    m = OracleModel(cfg, w)
    cache = KVCache(cfg, 64)
    lopa.prefill(m, cache, synth.prompt(cfg, 32).numpy(), 16)
    rng = np.random.default_rng(9)
    bt = np.where(rng.random((4, 16)) < 0.7, cfg["mask_id"], rng.integers(0, 1000, (4, 16)))
    bat = m.forward_block(bt, 32, cache)
    for j in range(4):
        one = m.forward_block(bt[j:j + 1], 32, cache)
        assert np.allclose(bat["conf"][j], one["conf"][0], rtol=1e-12, atol=1e-15)
        assert np.array_equal(bat["pred"][j], one["pred"][0])
        assert np.allclose(bat["k"][j], one["k"][0], atol=1e-13)


def test_faithful_close_to_pure():
    cfg, w = _tiny()
    mp, mf = OracleModel(cfg, w), OracleModel(cfg, w, "faithful")
    cp, cf = KVCache(cfg, 64), KVCache(cfg, 64)
    pr = synth.prompt(cfg, 32).numpy()
    lopa.prefill(mp, cp, pr, 16)
    lopa.prefill(mf, cf, pr, 16)
    blk = np.full((1, 16), cfg["mask_id"])
    a, b = mp.forward_block(blk, 32, cp), mf.forward_block(blk, 32, cf)
    assert np.max(np.abs(a["conf"] - b["conf"])) < 2e-2
    assert np.max(np.abs(cf.k[:, :, :32] - cp.k[:, :, :32])) < 0.05 * np.max(np.abs(cp.k))
    # faithful stores bf16 values
    assert np.array_equal(bf16_round(cf.k[:, :, :32]), cf.k[:, :, :32])


# ----------------------------------------------- bf16 rounding points (R16)
# The faithful mode rounds to bf16 exactly where a bf16 implementation stores
# a value: the input of every projection (h, o, h2, a and the final hf), q, k
# and v after bias / RoPE, and the softmax numerators p that multiply V (taken
# against the global row maximum). The residual stream x, the scores, the
# softmax sums and the logits stay unrounded.
ROUNDED = ("h", "q", "k", "v", "p", "o", "h2", "a")


def _trace(mode, P=24, L=16, nb=3, seed=5):
    cfg, w = _tiny()
    w = synth.to_bf16_values(w)
    m = OracleModel(cfg, w, mode)
    cache = KVCache(cfg, P + L)
    lopa.prefill(m, cache, synth.prompt(cfg, P).numpy(), L)
    rng = np.random.default_rng(seed)
    bt = np.where(rng.random((nb, L)) < 0.6, cfg["mask_id"], rng.integers(0, cfg["vocab"] - 1, (nb, L)))
    tr = []
    out = m.forward_block(bt, P, cache, trace=tr, keep_hidden=True)
    return cfg, tr, out


def _is_bf16(v):
    return np.array_equal(bf16_round(v), v)


def test_faithful_rounds_exactly_the_r16_points():
    cfg, tr, out = _trace("faithful")
    names = {}
    for name, li, v in tr:
        names.setdefault(name, set()).add(li)
        if name in ROUNDED or name == "hf":
            assert _is_bf16(v), f"{name} of layer {li} is not a bf16 value"
        elif name == "x":
            assert not _is_bf16(v), f"residual stream of layer {li} was rounded"
    layers = set(range(cfg["layers"]))
    for name in ROUNDED + ("x",):
        assert names.get(name) == layers, f"{name} not traced in every layer"
    assert names["hf"] == {cfg["layers"]}
    # the numerators are taken against the global row maximum: each row's
    # largest numerator is exactly exp(0) = 1
    for name, li, v in tr:
        if name == "p":
            assert np.array_equal(v.max(axis=-1), np.ones(v.shape[:-1]))
    # the logits are not rounded
    assert not _is_bf16(out["logits"])


def test_pure_rounds_nothing():
    """The same trace in the pure mode has no bf16 values at those points, so a
    rounding dropped from the faithful mode shows up in the test above."""
    cfg, tr, _ = _trace("pure")
    for name, li, v in tr:
        if name in ROUNDED + ("hf", "x") and name != "p":
            assert not _is_bf16(v), f"{name} of layer {li} is bf16 in the pure mode"
        if name == "p":
            off = v[v < 1.0]
            assert not _is_bf16(off)


def test_each_rounding_point_changes_the_result():
    """Dropping any single rounding point of the faithful mode changes its
    output (so every point is live, not only present in the trace)."""
    cfg, w = _tiny()
    w = synth.to_bf16_values(w)
    P, L = 24, 16
    base = OracleModel(cfg, w, "faithful")
    cache = KVCache(cfg, P + L)
    lopa.prefill(base, cache, synth.prompt(cfg, P).numpy(), L)
    bt = np.full((2, L), cfg["mask_id"])
    ref = base.forward_block(bt, P, cache, keep_hidden=True)
    for skip in ROUNDED + ("hf",):
        # every rounding goes through _store, in the order h, q, k, v, the
        # numerators of each head, o, h2, a per layer, then hf: count the calls
        # to check that order, then skip the one point under test
        m = OracleModel(cfg, w, "faithful")
        orig = m._store
        order = []

        def store(a, orig=orig, order=order):
            order.append(a.shape)
            return orig(a)
        m._store = store
        m.forward_block(bt, P, cache)
        heads = cfg["heads"]
        per_layer = ["h", "q", "k", "v"] + ["p"] * heads + ["o", "h2", "a"]
        seq = per_layer * cfg["layers"] + ["hf"]
        assert len(seq) == len(order)
        m2 = OracleModel(cfg, w, "faithful")
        it = iter(seq)

        def store2(a, it=it, skip=skip, orig=m2._store):
            return a if next(it) == skip else orig(a)
        m2._store = store2
        got = m2.forward_block(bt, P, cache, keep_hidden=True)
        assert not np.array_equal(got["logits"], ref["logits"]), f"dropping {skip} changes nothing"
