"""Pins of the oracle's decision rules (Eq. 1, Alg. 1 steps 1-3, Eq. 2, Conf).

Checks against hand-worked examples (tests/golden), exhaustive enumeration on
small grids, library special cases (numpy stable argsort, scipy logsumexp) and
the invariants the paper states (every branch fill set contains B0's)."""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import lopa
from oracle.model import confidence

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")))


def _f(v):
    return {"inf": math.inf, "-inf": -math.inf}.get(v, v) if isinstance(v, str) else v


@pytest.mark.parametrize("case", GOLD["eq1_and_branches"], ids=lambda c: c["cite"][:40])
def test_golden_branches(case):
    unfilled = np.array(case["tokens"]) == case["mask_id"]
    fill = lopa.threshold_fill(case["conf"], unfilled, case["tau"])
    assert sorted(fill.tolist()) == case["expect_fill"]
    bt, fp, valid, nv = lopa.build_branches(case["tokens"], case["conf"], case["pred"],
                                            case["mask_id"], case["tau"], case["k"])
    assert bt.tolist() == case["expect_branch_tokens"]
    assert fp.tolist() == case["expect_fill_pos"]
    assert valid.tolist() == case["expect_valid"]
    assert nv == case["expect_n_valid"]


@pytest.mark.parametrize("case", GOLD["eq2_select"], ids=lambda c: c["cite"][:40])
def test_golden_select(case):
    scores, w = lopa.select(np.array(case["branch_tokens"]), np.array(case["conf"]),
                            case["valid"], case["mask_id"])
    exp = [_f(v) for v in case["expect_scores"]]
    for s, e in zip(scores, exp):
        if math.isinf(e):
            assert s == e
        else:
            assert abs(s - e) < 1e-12
    assert w == case["expect_winner"]


@pytest.mark.parametrize("case", GOLD["confidence"], ids=lambda c: c["cite"][:40])
def test_golden_confidence(case):
    c, p = confidence(np.array(case["logits"])[None], case["mask_id"])
    assert abs(c[0] - case["expect_conf"]) < 1e-12
    assert p[0] == case["expect_pred"]


def test_eq1_exhaustive_grid():
    """All unfilled masks and conf vectors on a grid for L <= 5: I_fill is non-empty,
    inside M_t, equals S_high when S_high is non-empty, else is the single
    highest-conf unfilled position with the lowest index among ties."""
    grid = [0.1, 0.5, 0.9, 0.95]
    tau = 0.9
    for L in range(1, 6):
        for conf in itertools.product(grid, repeat=L):
            for um in itertools.product([0, 1], repeat=L):
                if not any(um):
                    continue
                f = set(lopa.threshold_fill(conf, um, tau).tolist())
                M = {i for i in range(L) if um[i]}
                assert f and f <= M
                high = {i for i in M if conf[i] > tau}
                if high:
                    assert f == high
                else:
                    (i,) = f
                    assert conf[i] == max(conf[j] for j in M)
                    assert all(conf[j] < conf[i] for j in M if j < i)


def test_topk_matches_stable_argsort():
    """Alg. 1 step 2 top-k == numpy's stable argsort of -conf restricted to M_B0."""
    rng = np.random.default_rng(5)
    mask = 99
    for _ in range(300):
        L = int(rng.integers(1, 33))
        conf = np.round(rng.random(L), 1)          # coarse values -> many ties
        tokens = np.where(rng.random(L) < 0.7, mask, rng.integers(0, 50, L))
        if not np.any(tokens == mask):
            continue
        pred = rng.integers(0, 50, L)
        k = int(rng.integers(0, 9))
        bt, fp, valid, nv = lopa.build_branches(tokens, conf, pred, mask, 0.85, k)
        b0 = bt[0]
        rem = np.flatnonzero(b0 == mask)
        order = np.argsort(-conf, kind="stable")
        ref = [int(i) for i in order if i in set(rem.tolist())][:k]
        assert fp[1:nv].tolist() == ref
        assert nv == 1 + min(k, len(rem))


def test_branch_invariants_random():
    """Every fill set contains B0's, has |I_fill|+1 fills, the p_j are distinct and
    avoid I_fill, padded branches equal B0, filled tokens are never the mask."""
    rng = np.random.default_rng(11)
    mask = 7
    for _ in range(300):
        L = int(rng.integers(1, 20))
        tokens = np.where(rng.random(L) < 0.8, mask, rng.integers(0, 7, L))
        if not np.any(tokens == mask):
            continue
        conf = rng.random(L)
        pred = rng.integers(0, 7, L)                 # never the mask id
        k = int(rng.integers(0, 6))
        tau = float(rng.choice([0.3, 0.9, 0.99]))
        bt, fp, valid, nv = lopa.build_branches(tokens, conf, pred, mask, tau, k)
        fill = set(lopa.threshold_fill(conf, tokens == mask, tau).tolist())
        orig_filled = set(np.flatnonzero(tokens != mask).tolist())
        b0_filled = set(np.flatnonzero(bt[0] != mask).tolist())
        assert b0_filled == orig_filled | fill
        ps = fp[1:nv].tolist()
        assert len(set(ps)) == len(ps) and not (set(ps) & fill)
        for j in range(bt.shape[0]):
            fj = set(np.flatnonzero(bt[j] != mask).tolist())
            assert fj >= b0_filled
            if valid[j] and j > 0:
                assert fj == b0_filled | {fp[j]}
                assert bt[j][fp[j]] == pred[fp[j]]
            if not valid[j]:
                assert np.array_equal(bt[j], bt[0]) and fp[j] == -1
        # tokens of the original filled positions never change
        assert np.all(bt[:, list(orig_filled)] == tokens[list(orig_filled)]) if orig_filled else True


def test_eq2_closed_form_and_permutation():
    rng = np.random.default_rng(3)
    mask = 5
    for _ in range(100):
        nb, L = int(rng.integers(1, 9)), int(rng.integers(1, 17))
        bt = np.where(rng.random((nb, L)) < 0.5, mask, 1)
        conf = rng.random((nb, L))
        valid = np.ones(nb, dtype=np.uint8)
        scores, w = lopa.select(bt, conf, valid, mask)
        for j in range(nb):
            m = bt[j] == mask
            ref = conf[j][m].mean() if m.any() else math.inf
            assert scores[j] == ref or abs(scores[j] - ref) < 1e-12
        # permuting branches permutes the scores; the winner's content is unchanged
        perm = rng.permutation(nb)
        s2, w2 = lopa.select(bt[perm], conf[perm], valid[perm], mask)
        assert np.allclose(s2, scores[perm], rtol=0, atol=1e-12) or np.array_equal(s2, scores[perm])
        assert np.array_equal(bt[perm][w2], bt[w]) or scores[perm][w2] == scores[w]


def test_identical_branches_identical_scores():
    bt = np.array([[5, 1, 5, 5]] * 4)
    conf = np.tile(np.array([0.3, 0.9, 0.2, 0.7]), (4, 1))
    scores, w = lopa.select(bt, conf, np.ones(4, np.uint8), 5)
    assert len(set(scores.tolist())) == 1 and w == 0


def test_confidence_softmax_properties():
    """conf == exp(max - logsumexp) over the support without the mask; probabilities
    sum to 1; conf in [1/(V-1), 1]; pred == first argmax."""
    rng = np.random.default_rng(0)
    for V in (2, 3, 17, 1000):
        lg = rng.normal(0, 6, (50, V))
        mask = V - 1
        conf, pred = confidence(lg, mask)
        sup = lg[:, :mask]
        ref = np.exp(sup.max(-1) - logsumexp(sup, axis=-1))
        assert np.allclose(conf, ref, rtol=1e-12, atol=0)
        p = np.exp(sup - logsumexp(sup, axis=-1, keepdims=True))
        assert np.allclose(p.sum(-1), 1.0, atol=1e-12)
        assert np.all(conf >= 1.0 / (V - 1) - 1e-15) and np.all(conf <= 1.0)
        assert np.array_equal(pred, np.argmax(sup, axis=-1))
        assert not np.any(pred == mask)


# ------------------------------------------- alternative branch confidences
def _rows(seed, n=300, L=12):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        conf = rng.random(L)
        tokens = np.where(rng.random(L) < 0.6, 7, rng.integers(0, 7, L))
        yield conf, tokens


def test_window_min_special_cases():
    """w = 1: the smallest unfilled Conf; w >= m: the Eq. 2 mean; m = 0: +inf;
    filled positions never matter."""
    for conf, tokens in _rows(0):
        un = tokens == 7
        if not un.any():
            assert lopa.branch_confidence_window_min(conf, tokens, 7, 3) == math.inf
            continue
        assert lopa.branch_confidence_window_min(conf, tokens, 7, 1) == pytest.approx(conf[un].min(), abs=0)
        m = int(un.sum())
        for w in (m, m + 1, 40):
            assert lopa.branch_confidence_window_min(conf, tokens, 7, w) == pytest.approx(
                lopa.branch_confidence(conf, tokens, 7), rel=1e-15)
        c2 = np.where(un, conf, 1.0 - conf)
        assert lopa.branch_confidence_window_min(c2, tokens, 7, 3) == \
            lopa.branch_confidence_window_min(conf, tokens, 7, 3)


def test_window_min_matches_convolution():
    """Library special case: the window means are a 'valid' convolution of the
    unfilled Conf sequence (position order) with a box of width w."""
    for conf, tokens in _rows(1):
        vals = conf[tokens == 7]
        for w in (2, 3, 5):
            if len(vals) < w:
                continue
            ref = np.convolve(vals, np.ones(w) / w, mode="valid").min()
            assert lopa.branch_confidence_window_min(conf, tokens, 7, w) == pytest.approx(ref, rel=1e-12)
            # reversing the position order gives the same windows
            assert lopa.branch_confidence_window_min(conf[::-1], tokens[::-1], 7, w) == \
                pytest.approx(ref, rel=1e-12)


def test_lowest_segment_properties():
    """eta = 1: the Eq. 2 mean; a tiny eta: the minimum; nondecreasing in eta,
    never above the mean; equal to the mean of np.partition's k smallest."""
    for conf, tokens in _rows(2):
        un = tokens == 7
        if not un.any():
            assert lopa.branch_confidence_lowest_segment(conf, tokens, 7, 0.5) == math.inf
            continue
        mean = lopa.branch_confidence(conf, tokens, 7)
        assert lopa.branch_confidence_lowest_segment(conf, tokens, 7, 1.0) == pytest.approx(mean, rel=1e-15)
        assert lopa.branch_confidence_lowest_segment(conf, tokens, 7, 1e-9) == conf[un].min()
        prev = -math.inf
        for eta in (0.1, 0.25, 0.5, 0.75, 1.0):
            v = lopa.branch_confidence_lowest_segment(conf, tokens, 7, eta)
            assert prev <= v + 1e-15 and v <= mean + 1e-15
            prev = v
            k = max(1, math.ceil(eta * un.sum()))
            assert v == pytest.approx(np.partition(conf[un], k - 1)[:k].mean(), rel=1e-12)


def test_select_with_metrics_invalid_and_ties():
    bt = np.array([[7, 7, 1, 7], [7, 7, 1, 7], [2, 7, 1, 7]])
    conf = np.array([[0.2, 0.9, 0.5, 0.4], [0.2, 0.9, 0.5, 0.4], [0.1, 0.3, 0.5, 0.3]])
    for metric in (lopa.METRIC_WINDOW_MIN, lopa.METRIC_LOWEST_SEGMENT):
        s, w = lopa.select(bt, conf, np.array([1, 1, 1], np.uint8), 7, metric, 2, 0.5)
        assert s[0] == s[1] and w == 0          # identical rows tie: lowest index
        s, w = lopa.select(bt, conf, np.array([0, 1, 1], np.uint8), 7, metric, 2, 0.5)
        assert s[0] == -math.inf and w == 1
    # hand-worked: unfilled Conf of row 0 in position order 0.2, 0.9, 0.4
    assert lopa.branch_score(conf[0], bt[0], 7, lopa.METRIC_WINDOW_MIN, 2, 0) == pytest.approx(0.55)
    assert lopa.branch_score(conf[0], bt[0], 7, lopa.METRIC_LOWEST_SEGMENT, 4, 0.5) == pytest.approx(0.3)
    assert lopa.branch_score(conf[2], bt[2], 7, lopa.METRIC_WINDOW_MIN, 2, 0) == pytest.approx(0.3)


def test_branches_with_eligible_prefix():
    """n_eligible = L is the plain rule; otherwise the threshold fill still uses
    every unfilled position while the fallback and the lookahead positions are
    the plain rule applied to the eligible prefix (checked on that prefix)."""
    rng = np.random.default_rng(5)
    for _ in range(400):
        L = int(rng.integers(2, 12))
        tokens = np.where(rng.random(L) < 0.7, 7, rng.integers(0, 7, L))
        n_el = int(rng.integers(1, L + 1))
        if not np.any(tokens[:n_el] == 7):
            tokens[rng.integers(n_el)] = 7
        conf = np.round(rng.random(L), 2)
        pred = rng.integers(0, 7, L)
        tau = float(rng.choice([0.3, 0.6, 0.95]))
        k = int(rng.integers(0, 4))
        a = lopa.build_branches(tokens, conf, pred, 7, tau, k)
        b = lopa.build_branches(tokens, conf, pred, 7, tau, k, L)
        assert all(np.array_equal(x, y) for x, y in zip(a[:3], b[:3])) and a[3] == b[3]
        bt, fp, valid, nv = lopa.build_branches(tokens, conf, pred, 7, tau, k, n_el)
        un = tokens == 7
        high = un & (conf > tau)
        b0 = bt[0]
        if high.any():
            assert np.array_equal(b0 != tokens, high)
        else:
            # fallback: the plain rule on the eligible prefix alone
            pb = lopa.build_branches(tokens[:n_el], conf[:n_el], pred[:n_el], 7, tau, k)
            assert np.array_equal(b0[:n_el], pb[0][0]) and np.array_equal(b0[n_el:], tokens[n_el:])
        assert np.all(fp[1:nv] < n_el) and np.all(fp[1:nv] >= 0)
        rem = [i for i in range(n_el) if b0[i] == 7]
        assert nv == 1 + min(k, len(rem))
