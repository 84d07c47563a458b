"""GPU parity of whole LoPA iterations (Alg. 1) and decoded blocks.

Teacher-forced: every iteration the GPU gets the oracle's state (block
tokens, confidences, candidates and the committed K/V cache) and the four
C-ABI calls are compared one by one. Free-running: the GPU decodes a block on
its own; at every iteration each of its decisions is checked against the
oracle's decision on the GPU's own inputs (Eq. 1 and the lookahead branches
from the GPU's state, the forward against the oracle forward of the same
branches, Eq. 2 and the winner from the GPU's confidences), so the whole
trajectory is a LoPA trajectory of the GPU's forward. The tolerances are the
fixed ones of gpu_util; a near-tie is a decision whose oracle margin is below
1e-3."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import (NEAR_TIE, conf_tol, Setup, check_forward, f32, log,
                      score_margin)
from oracle import lopa

pytestmark = pytest.mark.gpu

I32, F32, U8 = torch.int32, torch.float32, torch.uint8


def _d(a, dt):
    return torch.tensor(np.asarray(a), dtype=dt, device="cuda").contiguous()


@pytest.mark.parametrize("cfgname,P,L,k,tau", [("tiny", 64, 16, 3, 0.9), ("tiny", 64, 16, 7, 0.5),
                                               ("small", 100, 32, 7, 0.9), ("tiny", 40, 16, 3, 0.999)])
def test_teacher_forced_iterations(cfgname, P, L, k, tau):
    log(f"teacher-forced {cfgname} P={P} L={L} k={k} tau={tau}")
    s = Setup(cfgname, P, L, k)
    s.gpu_prefill()
    s.load_oracle_cache()
    lp, mask, nb = s.lp, s.cfg["mask_id"], k + 1
    tau32 = f32(tau)
    state = lopa.init_block(s.faith, s.cache_f, P, L)
    steps = checked = 0
    while (state[0] == mask).any():
        tokens, conf, pred = state
        conf32 = conf.astype(np.float32)
        # build on the oracle's state (conf as the fp32 values the GPU holds)
        bt = torch.empty(nb * L, dtype=I32, device="cuda")
        fp = torch.empty(nb, dtype=I32, device="cuda")
        va = torch.empty(nb, dtype=U8, device="cuda")
        nv = torch.empty(1, dtype=I32, device="cuda")
        lp.lopa_build_branches(_d(tokens, I32), _d(conf32, F32), _d(pred, I32), L, mask, tau, k,
                               bt, fp, va, nv)
        rbt, rfp, rva, rnv = lopa.build_branches(tokens, conf32.astype(np.float64), pred, mask, tau32, k)
        assert np.array_equal(bt.view(nb, L).cpu().numpy(), rbt)
        assert np.array_equal(va.cpu().numpy(), rva) and int(nv.item()) == rnv
        # verify the oracle's branches
        conf_b = torch.empty(nb * L, dtype=F32, device="cuda")
        pred_b = torch.empty(nb * L, dtype=I32, device="cuda")
        lp.lopa_verify_forward(s.model, s.kv, P, _d(rbt.ravel(), I32), nb, L, conf_b, pred_b)
        gc = conf_b.view(nb, L).cpu().numpy().astype(np.float64)
        gp = pred_b.view(nb, L).cpu().numpy()
        st = check_forward(s, rbt, gc, gp, label=f"iteration {steps}")
        # select on the GPU's verification outputs: the oracle's Eq. 2 on the
        # same confidences decides the winner; the scores also within the
        # end-to-end tolerance of the pure oracle's
        scores = torch.empty(nb, dtype=F32, device="cuda")
        win = torch.empty(1, dtype=I32, device="cuda")
        nt = torch.empty(L, dtype=I32, device="cuda")
        ncf = torch.empty(L, dtype=F32, device="cuda")
        npd = torch.empty(L, dtype=I32, device="cuda")
        nu = torch.empty(1, dtype=I32, device="cuda")
        lp.lopa_branch_confidence_select(_d(rbt.ravel(), I32), conf_b, pred_b, _d(rva, U8), nb, L,
                                         mask, scores, win, nt, ncf, npd, nu)
        gs = scores.cpu().numpy().astype(np.float64)
        ts, tw = lopa.select(rbt, gc, rva, mask)
        ps, _ = lopa.select(rbt, st["pure"]["conf"], rva, mask)
        fin = np.isfinite(ts)
        assert np.array_equal(np.isfinite(gs), fin) and np.array_equal(gs[~fin], ts[~fin])
        assert np.max(np.abs(gs[fin] - ts[fin]), initial=0) <= 1e-5
        assert np.max(np.abs(gs[fin] - ps[fin]), initial=0) <= conf_tol(s.cfg)
        w = int(win.item())
        if score_margin(ts) >= NEAR_TIE:
            assert np.array_equal(rbt[w], rbt[tw])
            checked += 1
        rw = lopa.select(rbt, st["faith"]["conf"], rva, mask)[1]
        # commit the oracle's winner and compare the written rows (and re-sync the
        # GPU prefix to the oracle's, as the next iteration is teacher-forced too)
        off = torch.empty(1, dtype=I32, device="cuda")
        lp.lopa_commit_kv(s.kv, _d([rw], I32), P, L, off)
        assert int(off.item()) == P
        for layer in range(s.cfg["layers"]):
            kk, vv = s.kv.read(layer, P, L)
            ref = st["faith"]["k"][rw, layer]
            assert np.max(np.abs(kk.float().cpu().numpy() - ref)) <= 0.05 * max(1.0, np.abs(ref).max())
        state, _ = lopa.lopa_step(s.faith, s.cache_f, P, state, k, tau32)
        s.load_oracle_cache(P + L)
        steps += 1
    log(f"  {steps} iterations, {checked} winners compared exactly")
    assert steps >= 1 and checked >= 1


def _first_divergence(gtrace, otrace):
    for t, (g, o) in enumerate(zip(gtrace, otrace)):
        gw = g["branch_tokens"][g["winner"]].numpy()
        ow = o["branch_tokens"][o["winner"]]
        if not np.array_equal(gw, ow):
            return t
    return None


# (config, P, L, k, tau, (metric, window, eta), fewest iterations): tau 0.999
# makes the blocks take many iterations (one or two fills each)
FREE = [("tiny", 64, 16, 3, 0.9, (0, 4, 0.25), 1), ("tiny", 32, 16, 0, 0.9, (0, 4, 0.25), 1),
        ("small", 100, 32, 7, 0.9, (0, 4, 0.25), 1), ("small128", 40, 16, 2, 0.7, (0, 4, 0.25), 1),
        ("tiny", 64, 16, 3, 0.9, (1, 4, 0.25), 1), ("tiny", 64, 16, 5, 0.9, (2, 4, 0.25), 1),
        ("tiny", 48, 16, 3, 0.999, (0, 4, 0.25), 4), ("small", 64, 32, 7, 0.999, (0, 4, 0.25), 4),
        ("tiny", 48, 16, 2, 0.999, (1, 3, 0.25), 4)]


@pytest.mark.parametrize("cfgname,P,L,k,tau,metric,min_iters", FREE)
def test_free_running_block(cfgname, P, L, k, tau, metric, min_iters):
    """metric = (branch confidence, window, eta): Eq. 2, or the window minimum /
    lowest-segment alternatives. The GPU decodes the block on its own (prefix
    K/V teacher-forced, so the oracle forward of each iteration sees the same
    prefix); every iteration is then replayed decision by decision."""
    log(f"free-running {cfgname} P={P} L={L} k={k} tau={tau} metric={metric}")
    s = Setup(cfgname, P, L, k)
    dec = s.gpu_prefill(tau)
    s.load_oracle_cache()
    dec.metric, dec.window, dec.eta = metric[0], metric[1], metric[2]
    gtrace = []
    g_iters = dec.decode_block(P, gtrace)
    mask, nb, tau32 = s.cfg["mask_id"], k + 1, f32(tau)
    g_tokens = dec.tokens.cpu().numpy()
    assert not np.any(g_tokens == mask) and len(gtrace) == g_iters >= min_iters
    excused = 0
    for t, g in enumerate(gtrace):
        tokens, conf, pred = (v.numpy() for v in g["state"])
        # Eq. 1 + lookahead branches from the GPU's own state (fp32 conf)
        rbt, rfp, rva, rnv = lopa.build_branches(tokens, conf.astype(np.float64), pred, mask, tau32, k)
        gbt = g["branch_tokens"].numpy()
        assert np.array_equal(gbt, rbt), f"iteration {t}: branches differ"
        assert np.array_equal(g["valid"].numpy(), rva) and g["n_valid"] == rnv
        # the verify forward of these branches against the oracle's
        gc = g["conf"].numpy().astype(np.float64)
        gp = g["pred"].numpy()
        st = check_forward(s, rbt, gc, gp, layers=t == 0, label=f"iteration {t}")
        # selection from the GPU's confidences; scores also vs the pure oracle's
        ts, tw = lopa.select(rbt, gc, rva, mask, metric[0], metric[1], f32(metric[2]))
        ps, _ = lopa.select(rbt, st["pure"]["conf"], rva, mask, metric[0], metric[1], f32(metric[2]))
        gs = g["scores"].numpy().astype(np.float64)
        fin = np.isfinite(ts)
        assert np.array_equal(np.isfinite(gs), fin) and np.array_equal(gs[~fin], ts[~fin])
        assert np.max(np.abs(gs[fin] - ts[fin]), initial=0) <= 1e-5
        assert np.max(np.abs(gs[fin] - ps[fin]), initial=0) <= conf_tol(s.cfg)
        if score_margin(ts) >= NEAR_TIE:
            assert np.array_equal(rbt[g["winner"]], rbt[tw]), f"iteration {t}: winner differs"
        else:
            excused += 1
        # the next state is the winner's row
        assert np.array_equal(g["tokens"].numpy(), rbt[g["winner"]])
    # the oracle's own trajectory (its own forwards): reported, not asserted --
    # two bf16 computations take different branches where a margin is within
    # their confidence difference
    otrace = []
    o_tokens, o_iters, _ = lopa.decode_block(s.faith, s.cache_f.copy(), P, L, k, tau32, otrace,
                                             metric[0], metric[1], f32(metric[2]))
    t = _first_divergence(gtrace, otrace)
    log(f"  {g_iters} iterations, {excused} winner near-ties; oracle's own trajectory: "
        + ("identical" if t is None and np.array_equal(g_tokens, o_tokens) else f"diverges at iteration {t}"))


# ---------------------------------------------- multi-block window (R27-R30)
WINDOW_CASES = [("tiny", 32, 16, 3, 0.9, 0.1, 0.5, 2, 48), ("tiny", 32, 16, 2, 0.9, 0.0, 0.3, 4, 64),
                ("small", 64, 32, 3, 0.9, 0.1, 0.5, 2, 64),
                # windows past 64 positions: 6 x 16, 4 x 32 and 8 x 32 (row groups of
                # the attention, 256-position build / select)
                ("tiny", 32, 16, 3, 0.9, 0.0, 0.3, 6, 96), ("small", 64, 32, 3, 0.9, 0.0, 0.5, 4, 128),
                ("small", 16, 32, 1, 0.9, 0.0, 0.5, 8, 256)]
FREE_WINDOW_CASES = [WINDOW_CASES[i] for i in (0, 1, 3, 4, 5)]
FORWARD_CHECKS_LONG = 6  # forwards compared with the oracle per long-window case


def _load_rows(s, cache, upto):
    for layer in range(s.cfg["layers"]):
        k = torch.tensor(cache.k[layer, :, :upto], dtype=torch.bfloat16, device="cuda")
        v = torch.tensor(cache.v[layer, :, :upto], dtype=torch.bfloat16, device="cuda")
        s.kv.write(layer, 0, k.contiguous(), v.contiguous())


@pytest.mark.parametrize("cfgname,P,L,k,tau,tau_add,tau_act,w_max,gen", WINDOW_CASES)
def test_window_teacher_forced(cfgname, P, L, k, tau, tau_add, tau_act, w_max, gen):
    """Every iteration of the oracle's multi-block window decode replayed on the
    GPU from the oracle's state (window tokens / conf / pred, eligible prefix,
    committed cache rows): lopa_build_branches_window bit-exact, the verify
    forward over the whole window within the faithful tolerance, the selection,
    and lopa_commit_kv_rows of the blocks that leave the window."""
    _window_teacher_forced(cfgname, P, L, k, tau, tau_add, tau_act, w_max, gen, False)


@pytest.mark.parametrize("cfgname,P,L,k,tau,tau_add,tau_act,w_max,gen", WINDOW_CASES)
def test_window_teacher_forced_block_causal(cfgname, P, L, k, tau, tau_add, tau_act, w_max, gen):
    """The same replay with the block-wise causal mask inside the window (the
    Ascend system's protocol, Sec. 3.4)."""
    _window_teacher_forced(cfgname, P, L, k, tau, tau_add, tau_act, w_max, gen, True)


def _window_teacher_forced(cfgname, P, L, k, tau, tau_add, tau_act, w_max, gen, block_causal):
    log(f"window teacher-forced {cfgname} P={P} L={L} k={k} w_max={w_max} tau_add={tau_add} "
        f"tau_act={tau_act} block_causal={block_causal}")
    s = Setup(cfgname, 0, L * w_max, k, max_len=P + gen)
    lp, mask, nb = s.lp, s.cfg["mask_id"], k + 1
    cblk = L if block_causal else 0
    s.kv.set_block_causal(cblk)
    tau32 = f32(tau)
    prompt = synth.prompt(s.cfg, P).numpy()
    otrace = []
    res = lopa.decode_window(s.faith, prompt, gen, L, k, tau32, tau_add, tau_act, w_max, trace=otrace,
                             block_causal=block_causal)
    assert len(res["tokens"]) == gen and not np.any(res["tokens"] == mask)
    cache = res["cache"]
    checked = windows = 0
    for t_idx, it in enumerate(otrace):
        P_t, (tokens, conf, pred), n_el = it["prefix_len"], it["state"], it["n_eligible"]
        Lw = len(tokens)
        windows += Lw > L
        _load_rows(s, cache, P_t)
        conf32 = conf.astype(np.float32)
        bt = torch.empty(nb * Lw, dtype=I32, device="cuda")
        fp = torch.empty(nb, dtype=I32, device="cuda")
        va = torch.empty(nb, dtype=U8, device="cuda")
        nv = torch.empty(1, dtype=I32, device="cuda")
        lp.lopa_build_branches_window(_d(tokens, I32), _d(conf32, F32), _d(pred, I32), Lw, n_el, mask,
                                      tau, k, bt, fp, va, nv)
        rbt, rfp, rva, rnv = lopa.build_branches(tokens, conf32.astype(np.float64), pred, mask, tau32, k, n_el)
        assert np.array_equal(bt.view(nb, Lw).cpu().numpy(), rbt)
        assert np.array_equal(va.cpu().numpy(), rva) and int(nv.item()) == rnv
        # the oracle's branches through the GPU forward over the whole window
        obt, n_valid = it["branch_tokens"], it["n_valid"]
        conf_b = torch.empty(nb * Lw, dtype=F32, device="cuda")
        pred_b = torch.empty(nb * Lw, dtype=I32, device="cuda")
        lp.lopa_verify_forward(s.model, s.kv, P_t, _d(obt.ravel(), I32), nb, Lw, conf_b, pred_b)
        gc = conf_b.view(nb, Lw).cpu().numpy().astype(np.float64)
        gp = pred_b.view(nb, Lw).cpu().numpy()
        # per-layer comparisons on the first two multi-block windows; for
        # windows past 64 positions the whole-forward checks on the first
        # FORWARD_CHECKS_LONG iterations (every decision is replayed below)
        if L * w_max <= 64 or t_idx < FORWARD_CHECKS_LONG:
            check_forward(s, obt, gc, gp, P=P_t, cache_f=cache, causal_blk=cblk,
                          layers=Lw > L and windows <= 2, label=f"window {Lw} rows, prefix {P_t}")
        scores = torch.empty(nb, dtype=F32, device="cuda")
        win = torch.empty(1, dtype=I32, device="cuda")
        nt = torch.empty(Lw, dtype=I32, device="cuda")
        ncf = torch.empty(Lw, dtype=F32, device="cuda")
        npd = torch.empty(Lw, dtype=I32, device="cuda")
        nu = torch.empty(1, dtype=I32, device="cuda")
        lp.lopa_branch_confidence_select(_d(obt.ravel(), I32), conf_b, pred_b, _d(it["valid"], U8), nb,
                                         Lw, mask, scores, win, nt, ncf, npd, nu)
        ts, tw = lopa.select(obt, gc, it["valid"], mask)
        if score_margin(ts) >= NEAR_TIE:
            assert np.array_equal(obt[int(win.item())], obt[tw])
            checked += 1
        c = it["committed_blocks"]
        if c:
            off = torch.empty(1, dtype=I32, device="cuda")
            lp.lopa_commit_kv_rows(s.kv, _d([it["winner"]], I32), P_t, Lw, c * L, off)
            assert int(off.item()) == P_t
            for layer in range(s.cfg["layers"]):
                kk, vv = s.kv.read(layer, P_t, c * L)
                ref = it["k"][it["winner"], layer][:, :c * L]
                assert np.max(np.abs(kk.float().cpu().numpy() - ref)) <= 0.05 * max(1.0, np.abs(ref).max())
    log(f"  {len(otrace)} iterations ({windows} over more than one block), {checked} winners compared")
    assert checked >= 1 and windows >= 1


@pytest.mark.parametrize("block_causal", [False, True])
@pytest.mark.parametrize("cfgname,P,L,k,tau,tau_add,tau_act,w_max,gen", FREE_WINDOW_CASES)
def test_window_decoder_free_running(cfgname, P, L, k, tau, tau_add, tau_act, w_max, gen, block_causal):
    """The GPU WindowDecoder end to end: a filled, committed sequence; the
    device gates (lopa_window_update / _commit) against the oracle's window
    bookkeeping (WindowGates) driven by the GPU's own selections; every
    iteration's decisions replayed; the oracle's trajectory logged."""
    log(f"window free-running {cfgname} P={P} L={L} k={k} w_max={w_max} block_causal={block_causal}")
    s = Setup(cfgname, 0, L * w_max, k, max_len=P + gen)
    mask = s.cfg["mask_id"]
    prompt = synth.prompt(s.cfg, P)
    dec = s.lp.WindowDecoder(s.model, s.kv, L, k, tau, tau_add, tau_act, w_max,
                             block_causal=block_causal)
    gtrace = []
    out = dec.decode(prompt, gen, gtrace)
    g_tokens = out["tokens"].numpy()
    assert len(g_tokens) == gen and not np.any(g_tokens == mask)
    assert out["forwards"] >= out["iterations"] >= gen // (L * w_max)
    # replay every iteration's decisions on the GPU's own inputs: the window
    # state it started from, its forward against the oracle forward of the
    # same branches over the GPU's own committed prefix (rows [0, P) never
    # change once committed), and the selection from its confidences
    from oracle import KVCache
    cache = KVCache(s.cfg, P + gen)
    end = P + gen
    for layer in range(s.cfg["layers"]):
        kk, vv = s.kv.read(layer, 0, end)
        cache.k[layer, :, :end] = kk.float().cpu().numpy()
        cache.v[layer, :, :end] = vv.float().cpu().numpy()
    cblk = L if block_causal else 0
    # the device gates: each iteration's window (prefix, length, eligible
    # positions, rows) and its committed blocks as the oracle's bookkeeping
    # gives them from the GPU's selections
    gates = lopa.WindowGates(L, w_max, gen // L, tau_add, tau_act, mask)
    wt, wc, wp = np.zeros(0, np.int64), np.zeros(0), np.zeros(0, np.int64)
    Pg, grown = P, 0
    for t, g in enumerate(gtrace):
        wt, wc, wp, opened = gates.fill(wt, wc, wp)
        assert g["initial_forward"] == opened, f"iteration {t}: initial forward"
        assert (g["prefix_len"], g["window_len"], g["n_eligible"]) == (Pg, len(wt), gates.eligible()), \
            f"iteration {t}: window"
        st_t, st_c, st_p = (v.numpy() for v in g["state"])
        assert np.array_equal(st_t, wt), f"iteration {t}: window tokens"
        if not opened:
            assert np.array_equal(st_c, wc.astype(np.float32)) and np.array_equal(st_p, wp)
        grown = max(grown, len(wt))
        sel = g["tokens"].numpy().astype(np.int64)
        w = g["winner"]
        c = gates.after_select(sel)
        assert g["committed_blocks"] == c, f"iteration {t}: committed blocks"
        wt = sel[c * L:]
        wc = g["conf"].numpy()[w, c * L:].astype(np.float64)
        wp = g["pred"].numpy()[w, c * L:].astype(np.int64)
        Pg += c * L
    assert gates.committed == gen // L and grown > L
    if tau_add == 0.0:  # the window fills at once: it reached its full length
        assert grown == L * min(w_max, gen // L)
    log(f"  device gates as the oracle's bookkeeping over {len(gtrace)} iterations; "
        f"longest window {grown} positions")
    excused = 0
    for t, g in enumerate(gtrace):
        tokens, conf, pred = (v.numpy() for v in g["state"])
        rbt, rfp, rva, rnv = lopa.build_branches(tokens, conf.astype(np.float64), pred, mask, f32(tau), k,
                                                 g["n_eligible"])
        assert np.array_equal(g["branch_tokens"].numpy(), rbt), f"iteration {t}: branches differ"
        assert np.array_equal(g["valid"].numpy(), rva) and g["n_valid"] == rnv
        gc = g["conf"].numpy().astype(np.float64)
        if L * w_max <= 64 or t < FORWARD_CHECKS_LONG:
            check_forward(s, rbt, gc, g["pred"].numpy(), P=g["prefix_len"], cache_f=cache,
                          causal_blk=cblk, layers=False, label=f"iteration {t}")
        ts, tw = lopa.select(rbt, gc, rva, mask)
        if score_margin(ts) >= NEAR_TIE:
            assert g["winner"] == tw or np.array_equal(rbt[g["winner"]], rbt[tw])
        else:
            excused += 1
        assert np.array_equal(g["tokens"].numpy(), rbt[g["winner"]])
    own = "not run (long window)"
    if L * w_max <= 64:  # the oracle's own trajectory, for the log
        res = lopa.decode_window(s.faith, prompt.numpy(), gen, L, k, f32(tau), tau_add, tau_act,
                                 w_max, block_causal=block_causal)
        own = "identical" if np.array_equal(g_tokens, res["tokens"]) else "differs"
    log(f"  {out['iterations']} iterations, {out['forwards']} forwards, TPF {out['tpf']:.2f}; "
        f"{excused} winner near-ties; oracle's own trajectory {own}")
