"""Oracle of the LoPA iteration (arXiv 2512.16229, Sec. 3.1-3.2, Alg. 1, Eq. 1-2).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py). Plain numpy / Python loops.

State of one active block: tokens [L] (a position is unfilled iff it holds
mask_id), conf [L] and pred [L] from the forward pass on exactly these tokens.

Readings of points the paper leaves open:
  * Conf / candidate: greedy token and its probability (model.py).
  * Eq. 1 compares strictly (conf > tau); every argmax picks the lowest index
    among equal values.
  * Top-k of Alg. 1 step 2: order by (conf descending, position ascending);
    k_eff = min(k, |M_B0|); the k - k_eff missing branches are copies of B0
    marked invalid (fill position -1) and can never win.
  * B_j = B0 plus position p_j filled with the candidate token pred[p_j] drawn
    from p_theta(.|x_t) (greedy), so every branch's fill set contains B0's.
  * Eq. 2 uses branch j's own verification forward, over M_{B_j}; an empty
    M_{B_j} scores +inf (the branch completes the block); invalid -> -inf.
  * Logit reuse (Sec. 3.2): the winner's verification conf / pred seed the next
    iteration, so each iteration costs one forward; a block costs one initial
    forward on the all-mask block plus one forward per iteration, including the
    iteration whose winner completes the block (its K/V are then exact).
"""
from __future__ import annotations

import math

import numpy as np

from .model import KVCache, OracleModel


# ----------------------------------------------------------------- Eq. 1
def threshold_fill(conf, unfilled, tau: float, n_eligible=None) -> np.ndarray:
    """I_fill: the unfilled positions with Conf > tau; if none, the single unfilled
    position of highest Conf (lowest position among ties).  Eq. 1.
    n_eligible: only positions below it may take the fallback (a multi-block
    window's fully activated blocks; reading R29)."""
    conf = np.asarray(conf, dtype=np.float64)
    n_el = len(conf) if n_eligible is None else n_eligible
    allc = [i for i in range(len(conf)) if unfilled[i]]
    high = [i for i in allc if conf[i] > tau]
    if high:
        return np.array(high, dtype=np.int64)
    cand = [i for i in allc if i < n_el]
    if not cand:
        raise ValueError("no eligible unfilled position")
    best = cand[0]
    for i in cand[1:]:
        if conf[i] > conf[best]:
            best = i
    return np.array([best], dtype=np.int64)


# ------------------------------------------------------- Alg. 1 steps 1-2
def build_branches(tokens, conf, pred, mask_id: int, tau: float, k: int, n_eligible=None):
    """Anchor B0 (Eq. 1 fill) and k lookahead branches (top-k of M_B0).
    n_eligible: the lookahead positions are taken below it only (R29).

    Returns (branch_tokens [k+1, L] int64, fill_pos [k+1] int64 (-1 for B0 and
    for padding), valid [k+1] uint8, n_valid)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    conf = np.asarray(conf, dtype=np.float64)
    pred = np.asarray(pred, dtype=np.int64)
    L = len(tokens)
    unfilled = tokens == mask_id
    b0 = tokens.copy()
    fill = threshold_fill(conf, unfilled, tau, n_eligible)
    b0[fill] = pred[fill]
    n_el = L if n_eligible is None else n_eligible
    rem = [i for i in range(n_el) if b0[i] == mask_id]         # eligible part of M_B0
    rem.sort(key=lambda i: (-conf[i], i))
    k_eff = min(k, len(rem))
    bt = np.tile(b0, (k + 1, 1))
    fill_pos = np.full(k + 1, -1, dtype=np.int64)
    valid = np.zeros(k + 1, dtype=np.uint8)
    valid[0] = 1
    for j in range(1, k_eff + 1):
        p = rem[j - 1]
        bt[j, p] = pred[p]
        fill_pos[j] = p
        valid[j] = 1
    return bt, fill_pos, valid, 1 + k_eff


# ----------------------------------------------------------------- Eq. 2
def branch_confidence(conf_row, tokens_row, mask_id: int) -> float:
    """C(B) = mean of Conf over the branch's still-unfilled positions.  Eq. 2.
    An empty unfilled set gives +inf (reading: such a branch completes the block)."""
    vals = [float(c) for c, t in zip(conf_row, tokens_row) if t == mask_id]
    if not vals:
        return math.inf
    return sum(vals) / len(vals)


# Alternative branch-confidence measures named after Eq. 2 (Sec. 3.2, "other
# methods"); the paper gives no formula, so these are readings:
#   * window minimum ("local quality"): the unfilled positions in position
#     order p_1 < ... < p_m, c_i = Conf(p_i); for a window size w, the means of
#     all runs of w consecutive c_i (one run over all of them if m < w); the
#     score is the smallest of these means;
#   * lowest segment ("weak links"): the mean of the ceil(eta m) smallest c_i
#     (at least one), 0 < eta <= 1.
# Both give +inf for m = 0, as Eq. 2 does.
METRIC_MEAN, METRIC_WINDOW_MIN, METRIC_LOWEST_SEGMENT = 0, 1, 2


def branch_confidence_window_min(conf_row, tokens_row, mask_id: int, window: int) -> float:
    """Smallest mean over runs of `window` consecutive unfilled positions."""
    if window < 1:
        raise ValueError("window must be >= 1")
    vals = [float(c) for c, t in zip(conf_row, tokens_row) if t == mask_id]
    m = len(vals)
    if m == 0:
        return math.inf
    if m < window:
        return sum(vals) / m
    best = math.inf
    for r in range(m - window + 1):
        best = min(best, sum(vals[r:r + window]) / window)
    return best


def branch_confidence_lowest_segment(conf_row, tokens_row, mask_id: int, eta: float) -> float:
    """Mean of the ceil(eta m) least confident unfilled positions (at least one)."""
    if not 0.0 < eta <= 1.0:
        raise ValueError("eta must be in (0, 1]")
    vals = sorted(float(c) for c, t in zip(conf_row, tokens_row) if t == mask_id)
    m = len(vals)
    if m == 0:
        return math.inf
    n = max(1, math.ceil(eta * m))
    return sum(vals[:n]) / n


def branch_score(conf_row, tokens_row, mask_id: int, metric: int = METRIC_MEAN,
                 window: int = 4, eta: float = 0.25) -> float:
    if metric == METRIC_MEAN:
        return branch_confidence(conf_row, tokens_row, mask_id)
    if metric == METRIC_WINDOW_MIN:
        return branch_confidence_window_min(conf_row, tokens_row, mask_id, window)
    if metric == METRIC_LOWEST_SEGMENT:
        return branch_confidence_lowest_segment(conf_row, tokens_row, mask_id, eta)
    raise ValueError(f"unknown metric {metric}")


def select(branch_tokens, conf, valid, mask_id: int, metric: int = METRIC_MEAN,
           window: int = 4, eta: float = 0.25):
    """Scores of all branches and B* = argmax (lowest branch index among ties)."""
    nb = len(branch_tokens)
    scores = np.empty(nb)
    for j in range(nb):
        scores[j] = (branch_score(conf[j], branch_tokens[j], mask_id, metric, window, eta)
                     if valid[j] else -math.inf)
    best = 0
    for j in range(1, nb):
        if scores[j] > scores[best]:
            best = j
    return scores, best


# ------------------------------------------------------------- iteration
def init_block(model: OracleModel, cache: KVCache, prefix_len: int, L: int):
    """All-mask block and its first forward: the state the first iteration reads."""
    tokens = np.full(L, model.cfg["mask_id"], dtype=np.int64)
    out = model.forward_block(tokens[None], prefix_len, cache)
    return tokens, out["conf"][0], out["pred"][0]


def lopa_step(model: OracleModel, cache: KVCache, prefix_len: int, state, k: int, tau: float,
              metric: int = METRIC_MEAN, window: int = 4, eta: float = 0.25):
    """One LoPA iteration (Alg. 1): build, verify in one pass, score, select, commit.
    metric / window / eta: the branch confidence (Eq. 2 or an alternative above).

    Returns (new_state, info).  info holds the branches, scores, winner, the
    verification outputs and the committed offset."""
    tokens, conf, pred = state
    mask_id = model.cfg["mask_id"]
    bt, fill_pos, valid, n_valid = build_branches(tokens, conf, pred, mask_id, tau, k)
    out = model.forward_block(bt[:n_valid], prefix_len, cache)
    nb = k + 1
    conf_b = np.zeros((nb, len(tokens)))
    pred_b = np.zeros((nb, len(tokens)), dtype=np.int64)
    conf_b[:n_valid], pred_b[:n_valid] = out["conf"], out["pred"]
    scores, w = select(bt, conf_b, valid, mask_id, metric, window, eta)
    off = cache.commit(prefix_len, out["k"][w], out["v"][w])
    new_state = (bt[w].copy(), conf_b[w].copy(), pred_b[w].copy())
    info = dict(branch_tokens=bt, fill_pos=fill_pos, valid=valid, n_valid=n_valid,
                conf=conf_b, pred=pred_b, scores=scores, winner=w, append_offset=off,
                kv=(out["k"], out["v"]))
    return new_state, info


def decode_block(model, cache, prefix_len: int, L: int, k: int, tau: float, trace=None,
                 metric: int = METRIC_MEAN, window: int = 4, eta: float = 0.25):
    """Decode one block to completion.  Returns (tokens, iterations, forwards)."""
    state = init_block(model, cache, prefix_len, L)
    forwards, iters = 1, 0
    mask_id = model.cfg["mask_id"]
    while True:
        state, info = lopa_step(model, cache, prefix_len, state, k, tau, metric, window, eta)
        forwards += 1
        iters += 1
        if trace is not None:
            trace.append(info)
        if not np.any(state[0] == mask_id):
            return state[0], iters, forwards
        if iters > L:
            raise RuntimeError("block did not complete in L iterations")


def prefill(model: OracleModel, cache: KVCache, prompt, L: int) -> int:
    """Block-causal prompt encoding in blocks of L (the last may be shorter):
    each block attends to the committed prefix and bidirectionally within itself,
    then its K/V are committed.  Returns the new prefix length."""
    prompt = np.asarray(prompt, dtype=np.int64)
    pos = 0
    while pos < len(prompt):
        blk = prompt[pos:pos + L]
        out = model.forward_block(blk[None], pos, cache)
        cache.commit(pos, out["k"][0], out["v"][0])
        pos += len(blk)
    return pos


def decode(model, prompt, gen_len: int, L: int, k: int, tau: float, max_len=None):
    """Prefill the prompt, then generate gen_len tokens (gen_len / L blocks)."""
    prompt = np.asarray(prompt, dtype=np.int64)
    cache = KVCache(model.cfg, max_len or (len(prompt) + gen_len))
    P = prefill(model, cache, prompt, L)
    out, iters, forwards = [], 0, 0
    for _ in range(gen_len // L):
        toks, it, fw = decode_block(model, cache, P, L, k, tau)
        out.append(toks)
        iters += it
        forwards += fw
        P += L
    gen = np.concatenate(out) if out else np.zeros(0, dtype=np.int64)
    return dict(tokens=gen, iterations=iters, forwards=forwards,
                tpf=(len(gen) / forwards) if forwards else 0.0, cache=cache)


# ------------------------------------------- multi-block window (Sec. 3.3)
# LoPA on D2F treats all active blocks as one window for branch exploration,
# with full attention inside the window (Sec. 3.3); the appendix's tables give
# the D2F gates tau_add and tau_act next to tau_conf but not their rules.
# Readings (the oracle and the GPU decoder follow both):
#   R27 window: up to w_max consecutive blocks of L after the committed prefix;
#       Eq. 1, the lookahead branches, the verify forward and Eq. 2 run over
#       all its positions at once.
#   R28 adding (tau_add): before an iteration, while the window holds fewer
#       than w_max blocks, blocks remain, and the last block's filled fraction
#       is >= tau_add, an all-mask block is appended; until a forward covers it
#       its positions carry Conf 0.
#   R29 activation (tau_act): the window's first block is fully activated;
#       block i becomes so once block i-1 is, block i has been covered by a
#       forward, and block i-1's filled fraction is >= tau_act. The Eq. 1
#       fallback and the lookahead positions are taken in the fully activated
#       blocks (a prefix of the window); the others fill only above tau.
#   R30 commit: after an iteration the leading blocks of the winner with no
#       unfilled position leave the window and their K/V (from that forward)
#       enter the prefix; an empty window takes a new block with one initial
#       forward, as a single block does.
class WindowGates:
    """The window bookkeeping of R27-R30, model-free: which blocks form the
    window, which are fully activated, when blocks join and leave. Driven by
    the window's tokens after each selection; the caller runs the forwards.
    (R29's coverage condition always holds where it is tested: every block in
    the window at a selection was covered by that selection's forward.)"""

    def __init__(self, L: int, w_max: int, n_blocks: int, tau_add: float, tau_act: float,
                 mask_id: int):
        self.L, self.w_max, self.n_blocks = L, w_max, n_blocks
        self.tau_add, self.tau_act, self.mask_id = tau_add, tau_act, mask_id
        self.active, self.added, self.committed = [], 0, 0

    def filled(self, tokens, b) -> float:
        return float(np.mean(tokens[b * self.L:(b + 1) * self.L] != self.mask_id))

    def eligible(self) -> int:
        """Positions of the fully activated leading blocks (R29)."""
        return self.L * next((i for i, a in enumerate(self.active) if not a), len(self.active))

    def fill(self, tokens, conf, pred):
        """R27 / R30: an empty window with blocks left opens one (fully
        activated; its initial forward is due), then blocks are appended while
        the window has room, blocks remain and the last block is at least
        tau_add filled. Returns (tokens, conf, pred, opened)."""
        L, m = self.L, self.mask_id

        def append():
            nonlocal tokens, conf, pred
            tokens = np.concatenate([tokens, np.full(L, m, dtype=np.int64)])
            conf = np.concatenate([conf, np.zeros(L)])
            pred = np.concatenate([pred, np.full(L, m, dtype=np.int64)])
            self.active.append(len(self.active) == 0)
            self.added += 1

        opened = False
        if not self.active and self.added < self.n_blocks:
            append()
            opened = True
        while (len(self.active) < self.w_max and self.added < self.n_blocks
               and self.filled(tokens, len(self.active) - 1) >= self.tau_add):
            append()
        return tokens, conf, pred, opened

    def after_select(self, tokens):
        """R29 / R30 after a selection over the window: activation in block
        order, then c = the leading blocks with no unfilled position, which
        leave (the new first block is fully activated). Returns c; the caller
        commits their K/V and drops their rows."""
        for i in range(1, len(self.active)):
            if not self.active[i] and self.active[i - 1] and self.filled(tokens, i - 1) >= self.tau_act:
                self.active[i] = True
        c = 0
        while c < len(self.active) and not np.any(tokens[c * self.L:(c + 1) * self.L] == self.mask_id):
            c += 1
        if c:
            del self.active[:c]
            if self.active:
                self.active[0] = True
            self.committed += c
        return c


def decode_window(model: OracleModel, prompt, gen_len: int, L: int, k: int, tau: float,
                  tau_add: float, tau_act: float, w_max: int, metric: int = METRIC_MEAN,
                  window: int = 4, eta: float = 0.25, trace=None, max_len=None,
                  block_causal: bool = False):
    """Generate gen_len tokens (gen_len / L blocks) with a sliding window of up
    to w_max active blocks. Returns tokens, iterations, forwards, tpf, cache.
    block_causal: the window's blocks attend block-causally (a block sees the
    prefix, the earlier window blocks and itself; Sec. 3.4, LoPA-Dist-Ascend)
    instead of with full attention inside the window."""
    cblk = L if block_causal else 0
    mask_id = model.cfg["mask_id"]
    prompt = np.asarray(prompt, dtype=np.int64)
    cache = KVCache(model.cfg, max_len or (len(prompt) + gen_len))
    P = prefill(model, cache, prompt, L)
    n_blocks = gen_len // L
    gates = WindowGates(L, w_max, n_blocks, tau_add, tau_act, mask_id)
    tokens = np.zeros(0, dtype=np.int64)
    conf = np.zeros(0)
    pred = np.zeros(0, dtype=np.int64)
    out, iters, forwards = [], 0, 0

    while gates.committed < n_blocks:
        tokens, conf, pred, opened = gates.fill(tokens, conf, pred)
        if opened:
            # the new block's initial forward (the block alone)
            o = model.forward_block(tokens[None, :L], P, cache, causal_blk=cblk)
            conf[:L], pred[:L] = o["conf"][0], o["pred"][0]
            forwards += 1
        n_el = gates.eligible()
        state_in = (tokens.copy(), conf.copy(), pred.copy())
        bt, fill_pos, valid, n_valid = build_branches(tokens, conf, pred, mask_id, tau, k, n_el)
        o = model.forward_block(bt[:n_valid], P, cache, causal_blk=cblk)
        nb, Lw = k + 1, len(tokens)
        conf_b = np.zeros((nb, Lw))
        pred_b = np.zeros((nb, Lw), dtype=np.int64)
        conf_b[:n_valid], pred_b[:n_valid] = o["conf"], o["pred"]
        scores, w = select(bt, conf_b, valid, mask_id, metric, window, eta)
        forwards += 1
        iters += 1
        tokens, conf, pred = bt[w].copy(), conf_b[w].copy(), pred_b[w].copy()
        c = gates.after_select(tokens)
        if trace is not None:
            trace.append(dict(prefix_len=P, state=state_in, branch_tokens=bt, valid=valid,
                              n_valid=n_valid, n_eligible=n_el, conf=conf_b, pred=pred_b,
                              scores=scores, winner=w, committed_blocks=c, k=o["k"], v=o["v"]))
        if c:
            cache.commit(P, o["k"][w][:, :, :c * L], o["v"][w][:, :, :c * L])
            out.append(tokens[:c * L].copy())
            tokens, conf, pred = tokens[c * L:], conf[c * L:], pred[c * L:]
            P += c * L
        if iters > 2 * gen_len + 2 * n_blocks:
            raise RuntimeError("window decode did not converge")
    gen = np.concatenate(out) if out else np.zeros(0, dtype=np.int64)
    return dict(tokens=gen, iterations=iters, forwards=forwards,
                tpf=(len(gen) / forwards) if forwards else 0.0, cache=cache)


# ------------------------------------------- multi-block window (Sec. 3.3)
# LoPA on D2F treats all active blocks as one window for branch exploration,
# with full attention inside the window (Sec. 3.3); the appendix's tables give
# the D2F gates tau_add and tau_act next to tau_conf but not their rules.
# Readings (the oracle and the GPU decoder follow both):
#   R27 window: up to w_max consecutive blocks of L after the committed prefix;
#       Eq. 1, the lookahead branches, the verify forward and Eq. 2 run over
#       all its positions at once.
#   R28 adding (tau_add): before an iteration, while the window holds fewer
#       than w_max blocks, blocks remain, and the last block's filled fraction
#       is >= tau_add, an all-mask block is appended; until a forward covers it
#       its positions carry Conf 0.
#   R29 activation (tau_act): the window's first block is fully activated;
#       block i becomes so once block i-1 is, block i has been covered by a
#       forward, and block i-1's filled fraction is >= tau_act. The Eq. 1
#       fallback and the lookahead positions are taken in the fully activated
#       blocks (a prefix of the window); the others fill only above tau.
#   R30 commit: after an iteration the leading blocks of the winner with no
#       unfilled position leave the window and their K/V (from that forward)
#       enter the prefix; an empty window takes a new block with one initial
#       forward, as a single block does.
def decode_window(model: OracleModel, prompt, gen_len: int, L: int, k: int, tau: float,
                  tau_add: float, tau_act: float, w_max: int, metric: int = METRIC_MEAN,
                  window: int = 4, eta: float = 0.25, trace=None, max_len=None,
                  block_causal: bool = False):
    """Generate gen_len tokens (gen_len / L blocks) with a sliding window of up
    to w_max active blocks. Returns tokens, iterations, forwards, tpf, cache.
    block_causal: the window's blocks attend block-causally (a block sees the
    prefix, the earlier window blocks and itself; Sec. 3.4, LoPA-Dist-Ascend)
    instead of with full attention inside the window."""
    cblk = L if block_causal else 0
    mask_id = model.cfg["mask_id"]
    prompt = np.asarray(prompt, dtype=np.int64)
    cache = KVCache(model.cfg, max_len or (len(prompt) + gen_len))
    P = prefill(model, cache, prompt, L)
    n_blocks = gen_len // L
    tokens = np.zeros(0, dtype=np.int64)
    conf = np.zeros(0)
    pred = np.zeros(0, dtype=np.int64)
    active, covered = [], []
    out, added, committed, iters, forwards = [], 0, 0, 0, 0

    def filled_frac(b):
        return float(np.mean(tokens[b * L:(b + 1) * L] != mask_id))

    def append_block():
        nonlocal tokens, conf, pred, added
        tokens = np.concatenate([tokens, np.full(L, mask_id, dtype=np.int64)])
        conf = np.concatenate([conf, np.zeros(L)])
        pred = np.concatenate([pred, np.full(L, mask_id, dtype=np.int64)])
        active.append(len(active) == 0)
        covered.append(False)
        added += 1

    while committed < n_blocks:
        if not active:
            append_block()
            o = model.forward_block(tokens[None], P, cache, causal_blk=cblk)
            conf, pred = o["conf"][0].copy(), o["pred"][0].copy()
            covered[:] = [True] * len(covered)
            forwards += 1
        while len(active) < w_max and added < n_blocks and filled_frac(len(active) - 1) >= tau_add:
            append_block()
        n_el = L * next((i for i, a in enumerate(active) if not a), len(active))
        state_in = (tokens.copy(), conf.copy(), pred.copy())
        bt, fill_pos, valid, n_valid = build_branches(tokens, conf, pred, mask_id, tau, k, n_el)
        o = model.forward_block(bt[:n_valid], P, cache, causal_blk=cblk)
        nb, Lw = k + 1, len(tokens)
        conf_b = np.zeros((nb, Lw))
        pred_b = np.zeros((nb, Lw), dtype=np.int64)
        conf_b[:n_valid], pred_b[:n_valid] = o["conf"], o["pred"]
        scores, w = select(bt, conf_b, valid, mask_id, metric, window, eta)
        forwards += 1
        iters += 1
        tokens, conf, pred = bt[w].copy(), conf_b[w].copy(), pred_b[w].copy()
        covered[:] = [True] * len(covered)
        for i in range(1, len(active)):
            if not active[i] and active[i - 1] and covered[i] and filled_frac(i - 1) >= tau_act:
                active[i] = True
        c = 0
        while c < len(active) and not np.any(tokens[c * L:(c + 1) * L] == mask_id):
            c += 1
        if trace is not None:
            trace.append(dict(prefix_len=P, state=state_in, branch_tokens=bt, valid=valid,
                              n_valid=n_valid, n_eligible=n_el, conf=conf_b, pred=pred_b,
                              scores=scores, winner=w, committed_blocks=c, k=o["k"], v=o["v"]))
        if c:
            cache.commit(P, o["k"][w][:, :, :c * L], o["v"][w][:, :, :c * L])
            out.append(tokens[:c * L].copy())
            tokens, conf, pred = tokens[c * L:], conf[c * L:], pred[c * L:]
            del active[:c], covered[:c]
            if active:
                active[0] = True
            P += c * L
            committed += c
        if iters > 2 * gen_len + 2 * n_blocks:
            raise RuntimeError("window decode did not converge")
    gen = np.concatenate(out) if out else np.zeros(0, dtype=np.int64)
    return dict(tokens=gen, iterations=iters, forwards=forwards,
                tpf=(len(gen) / forwards) if forwards else 0.0, cache=cache)
