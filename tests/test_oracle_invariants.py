"""Invariants of the whole LoPA iteration on the oracle (Alg. 1, Eq. 1-2, Sec. 3.2).

* k = 0 reduces to plain confidence-threshold decoding (Eq. 1 alone).
* Brute force on a tiny vocab / block: with k >= |M_B0| the winner equals the
  best, by Eq. 2, of B0 and every one-position extension of B0, each forwarded
  on its own.
* Termination within L iterations; each iteration fills |I_fill| or |I_fill|+1.
* Identical branches get identical scores; permuting the verify batch permutes
  the outputs and leaves the winner's content unchanged.
* Resuming from a saved state (tokens, conf, pred, cache) replays the same
  trajectory."""
import copy
import math

import numpy as np
import pytest

import synth
from oracle import KVCache, OracleModel, lopa


@pytest.fixture(scope="module")
def tiny():
    cfg = synth.config("tiny")
    w = synth.model_weights(cfg)
    m = OracleModel(cfg, w)
    cache = KVCache(cfg, 64 + 64)
    P = lopa.prefill(m, cache, synth.prompt(cfg, 64).numpy(), 16)
    return cfg, m, cache, P


def threshold_decode(model, cache, P, L, tau):
    """Plain confidence-threshold decoding of one block (Eq. 1 on the current state)."""
    mask = model.cfg["mask_id"]
    x = np.full(L, mask)
    steps = 0
    while (x == mask).any():
        o = model.forward_block(x[None], P, cache)
        c, p = o["conf"][0], o["pred"][0]
        M = np.flatnonzero(x == mask)
        hi = M[c[M] > tau]
        fill = hi if hi.size else M[[np.argmax(c[M])]]
        x = x.copy()
        x[fill] = p[fill]
        steps += 1
    return x, steps


@pytest.mark.parametrize("tau", [0.9, 0.5, 0.2])
def test_k0_is_threshold_decoding(tiny, tau):
    cfg, m, cache, P = tiny
    ref, steps = threshold_decode(m, cache.copy(), P, 16, tau)
    toks, iters, forwards = lopa.decode_block(m, cache.copy(), P, 16, 0, tau)
    assert np.array_equal(toks, ref)
    assert iters == steps
    assert forwards == steps + 1          # + the verify forward of the completing branch


def test_termination_and_fill_growth(tiny):
    cfg, m, cache, P = tiny
    for k, tau in [(3, 0.9), (7, 0.5), (1, 0.99)]:
        trace = []
        toks, iters, fw = lopa.decode_block(m, cache.copy(), P, 16, k, tau, trace)
        assert iters <= 16 and fw == iters + 1
        mask = cfg["mask_id"]
        filled_before = 0
        for info in trace:
            bt, w = info["branch_tokens"], info["winner"]
            n0 = int((bt[0] != mask).sum())
            nw = int((bt[w] != mask).sum())
            assert nw in (n0, n0 + 1) and nw > filled_before
            filled_before = nw
        assert not np.any(toks == mask)


def test_brute_force_one_step_lookahead():
    """V = 16, L = 4, one layer, k >= |M_B0|: LoPA's winner is the Eq. 2 argmax over
    B0 and all single-position extensions of B0, each forwarded separately."""
    cfg = synth.config("tiny", layers=1, vocab=16, lm_std=2.0)
    w = synth.model_weights(cfg)
    m = OracleModel(cfg, w)
    cache = KVCache(cfg, 16)
    P = lopa.prefill(m, cache, synth.prompt(cfg, 8).numpy(), 4)
    mask = cfg["mask_id"]
    checked = 0
    for tau in (0.95, 0.6, 0.3):
        state = lopa.init_block(m, cache, P, 4)
        while (state[0] == mask).any():
            tokens, conf, pred = state
            new_state, info = lopa.lopa_step(m, cache.copy(), P, state, k=4, tau=tau)
            b0 = info["branch_tokens"][0]
            cands = [b0]
            for p in np.flatnonzero(b0 == mask):
                c = b0.copy()
                c[p] = pred[p]
                cands.append(c)
            best, best_s = None, -math.inf
            for c in cands:
                o = m.forward_block(c[None], P, cache)
                s = lopa.branch_confidence(o["conf"][0], c, mask)
                if s > best_s:
                    best, best_s = c, s
            assert np.array_equal(new_state[0], best)
            assert info["scores"][info["winner"]] == pytest.approx(best_s, rel=1e-12) \
                or (math.isinf(best_s) and math.isinf(info["scores"][info["winner"]]))
            state = new_state
            checked += 1
    assert checked >= 3


def test_identical_and_permuted_branches(tiny):
    cfg, m, cache, P = tiny
    mask = cfg["mask_id"]
    state = lopa.init_block(m, cache, P, 16)
    bt, fp, valid, nv = lopa.build_branches(*state, mask, 0.9, 5)
    out = m.forward_block(bt, P, cache)
    # identical branches (padding copies, or B0 duplicated) -> identical scores
    dup = np.stack([bt[0]] * 3)
    od = m.forward_block(dup, P, cache)
    sd, wd = lopa.select(dup, od["conf"], np.ones(3, np.uint8), mask)
    assert abs(sd[0] - sd[1]) < 1e-12 and abs(sd[1] - sd[2]) < 1e-12 and wd == 0
    # permutation of the batch
    perm = np.random.default_rng(1).permutation(len(bt))
    op = m.forward_block(bt[perm], P, cache)
    assert np.allclose(op["conf"], out["conf"][perm], atol=1e-12)
    s1, w1 = lopa.select(bt, out["conf"], valid, mask)
    s2, w2 = lopa.select(bt[perm], op["conf"], valid[perm], mask)
    assert np.array_equal(bt[perm][w2], bt[w1])


def test_resume_from_saved_state(tiny):
    cfg, m, cache, P = tiny
    c1 = cache.copy()
    trace = []
    ref, _, _ = lopa.decode_block(m, c1, P, 16, 3, 0.9, trace)
    # replay: stop after two iterations, save, restore into fresh objects, continue
    c2 = cache.copy()
    state = lopa.init_block(m, c2, P, 16)
    for _ in range(2):
        state, _ = lopa.lopa_step(m, c2, P, state, 3, 0.9)
    saved = copy.deepcopy((state, c2.k, c2.v))
    c3 = cache.copy()
    (state3, k3, v3) = saved
    c3.k[:], c3.v[:] = k3, v3
    while (state3[0] == cfg["mask_id"]).any():
        state3, _ = lopa.lopa_step(m, c3, P, state3, 3, 0.9)
    assert np.array_equal(state3[0], ref)
    assert np.array_equal(c3.k, c1.k) and np.array_equal(c3.v, c1.v)


def test_commit_writes_only_the_winner(tiny):
    """The committed rows equal the winner's block K/V; a poisoned loser never lands."""
    cfg, m, cache, P = tiny
    c = cache.copy()
    state = lopa.init_block(m, c, P, 16)
    new_state, info = lopa.lopa_step(m, c, P, state, 3, 0.9)
    k, v = info["kv"]
    w = info["winner"]
    assert np.array_equal(c.k[:, :, P:P + 16], k[w]) and info["append_offset"] == P
    assert not np.isnan(c.k).any()


def test_decode_small_end_to_end():
    """Prefill + 2 blocks on the tiny config; TPF = tokens / forwards >= 1."""
    cfg = synth.config("tiny")
    m = OracleModel(cfg, synth.model_weights(cfg))
    r = lopa.decode(m, synth.prompt(cfg, 64).numpy(), 32, 16, 3, 0.9)
    assert len(r["tokens"]) == 32 and not np.any(r["tokens"] == cfg["mask_id"])
    assert r["forwards"] == r["iterations"] + 2
    assert r["tpf"] >= 1.0


# ------------------------------------------- multi-block window (R27-R30)
@pytest.mark.parametrize("k,tau", [(3, 0.9), (0, 0.9), (5, 0.5)])
def test_window_of_one_block_is_block_decoding(k, tau):
    """w_max = 1, or a tau_add no fill fraction reaches, leaves one block in the
    window: the same tokens, iterations and forwards as block-by-block decoding."""
    cfg = synth.config("tiny")
    m = OracleModel(cfg, synth.model_weights(cfg), "faithful")
    prompt = synth.prompt(cfg, 32).numpy()
    ref = lopa.decode(m, prompt, 48, 16, k, tau)
    for w_max, tau_add in ((1, 0.1), (3, 1.5)):
        got = lopa.decode_window(m, prompt, 48, 16, k, tau, tau_add, 0.5, w_max)
        assert np.array_equal(got["tokens"], ref["tokens"])
        assert got["iterations"] == ref["iterations"] and got["forwards"] == ref["forwards"]
        assert np.array_equal(got["cache"].k, ref["cache"].k)


@pytest.mark.parametrize("w_max,tau_add,tau_act", [(2, 0.1, 0.5), (4, 0.0, 0.3), (3, 0.2, 0.95)])
def test_window_invariants(w_max, tau_add, tau_act):
    """Every generated position filled; blocks committed whole and in order;
    every iteration fills at least one position; the window never exceeds
    w_max blocks; the fallback and lookahead fills stay in the fully activated
    prefix; a committed block's K/V equal the forward that completed it."""
    cfg = synth.config("tiny")
    m = OracleModel(cfg, synth.model_weights(cfg), "faithful")
    mask, L, gen = cfg["mask_id"], 16, 64
    prompt = synth.prompt(cfg, 32).numpy()
    trace = []
    res = lopa.decode_window(m, prompt, gen, L, 3, 0.9, tau_add, tau_act, w_max, trace=trace)
    assert len(res["tokens"]) == gen and not np.any(res["tokens"] == mask)
    assert res["forwards"] >= res["iterations"]
    P = 32
    for it in trace:
        tokens, conf, pred = it["state"]
        Lw, n_el = len(tokens), it["n_eligible"]
        assert Lw % L == 0 and Lw <= w_max * L and n_el % L == 0 and L <= n_el <= Lw
        assert it["prefix_len"] == P
        w = it["winner"]
        new = it["branch_tokens"][w]
        filled = np.flatnonzero((tokens == mask) & (new != mask))
        assert filled.size >= 1
        # fills outside the eligible prefix come from the threshold only
        outside = filled[filled >= n_el]
        assert np.all(conf[outside] > 0.9)
        c = it["committed_blocks"]
        assert not np.any(new[:c * L] == mask)
        if c:
            assert np.array_equal(res["cache"].k[:, :, P:P + c * L], it["k"][w][:, :, :c * L])
        P += c * L
    assert P == 32 + gen


# ----------------------------- block-causal window (Sec. 3.4, LoPA-Dist-Ascend)
def test_block_causal_rows_match_block_forwards(tiny):
    """With the block-wise causal mask, the rows of window sub-block 0 are the
    forward of sub-block 0 alone, and the rows of sub-block 1 are the forward of
    sub-block 1 alone after sub-block 0's K/V were written to the cache at its
    positions (the pre-written K/V are final: no later block changes them).
    With a sub-block as long as the window the mask is no mask at all."""
    cfg, m, cache, P = tiny
    mask, L = cfg["mask_id"], 8
    rng = np.random.default_rng(11)
    bt = np.where(rng.random((3, 2 * L)) < 0.5, mask, rng.integers(0, cfg["vocab"] - 1, (3, 2 * L)))
    full = m.forward_block(bt, P, cache, causal_blk=L)
    first = m.forward_block(bt[:, :L], P, cache)
    np.testing.assert_allclose(full["conf"][:, :L], first["conf"], rtol=0, atol=1e-12)
    assert np.array_equal(full["pred"][:, :L], first["pred"])
    np.testing.assert_allclose(full["k"][..., :L, :], first["k"], rtol=0, atol=1e-10)
    np.testing.assert_allclose(full["v"][..., :L, :], first["v"], rtol=0, atol=1e-10)
    for j in range(3):
        c = cache.copy()
        c.commit(P, first["k"][j], first["v"][j])
        second = m.forward_block(bt[j:j + 1, L:], P + L, c)
        np.testing.assert_allclose(full["conf"][j, L:], second["conf"][0], rtol=0, atol=1e-12)
        assert np.array_equal(full["pred"][j, L:], second["pred"][0])
        np.testing.assert_allclose(full["k"][j][..., L:, :], second["k"][0], rtol=0, atol=1e-10)
    nomask = m.forward_block(bt, P, cache)
    same = m.forward_block(bt, P, cache, causal_blk=2 * L)
    assert np.array_equal(nomask["conf"], same["conf"]) and np.array_equal(nomask["k"], same["k"])
    # and the mask does change rows of sub-block 0 when later rows may be seen
    assert np.max(np.abs(nomask["conf"][:, :L] - full["conf"][:, :L])) > 0


@pytest.mark.parametrize("w_max,tau_add,tau_act", [(2, 0.1, 0.5), (3, 0.0, 0.3)])
def test_block_causal_window_cache_is_prefill_of_output(w_max, tau_add, tau_act):
    """Single-phase consistency: with block-causal attention in the window, the
    K/V a block leaves in the cache depend only on the prefix and the block's
    own final tokens, so the cache after the decode equals a block-causal
    prefill of prompt + generated tokens (prompt a whole number of blocks)."""
    cfg = synth.config("tiny")
    m = OracleModel(cfg, synth.model_weights(cfg), "faithful")
    mask, L, gen = cfg["mask_id"], 16, 64
    prompt = synth.prompt(cfg, 32).numpy()
    res = lopa.decode_window(m, prompt, gen, L, 3, 0.9, tau_add, tau_act, w_max, block_causal=True)
    assert len(res["tokens"]) == gen and not np.any(res["tokens"] == mask)
    ref = KVCache(cfg, 32 + gen)
    lopa.prefill(m, ref, np.concatenate([prompt, res["tokens"]]), L)
    np.testing.assert_allclose(res["cache"].k, ref.k, rtol=0, atol=1e-9)
    np.testing.assert_allclose(res["cache"].v, ref.v, rtol=0, atol=1e-9)
