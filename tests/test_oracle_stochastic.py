"""Pins of the stochastic prefix verifier oracle (Sec. III-D "Prefix verifier",
temperature T > 0).

References independent of the oracle: a hand-worked three-token example;
the distributions the procedure must produce, computed in closed form from
scipy's softmax and checked with chi-square tests over many uniforms -- the
first emitted token must follow the target distribution P of the anchor row
(the verifier is lossless), the accepted length must follow the product of
the candidates' probabilities, and after a rejection the successor must
follow P without the rejected candidate; and the greedy oracle in the
low-temperature limit.
"""
import numpy as np
import pytest
from scipy.special import softmax
from scipy.stats import chisquare

import oracle

P_MIN = 1e-4  # chi-square p-value floor (seeded draws: deterministic)


def test_hand_example():
    # P = [1/6, 2/6, 3/6] at T = 1; candidate x = 2 has P(x) = 1/2
    L = np.log(np.array([[1, 2, 3], [1, 2, 3]], np.float64)).astype(np.float32)
    cu = np.array([0, 2], np.int32)
    draft = np.array([7, 2], np.int32)
    cases = [((0.4, 0.3), (1, 1)),   # accepted; all passed -> P unchanged: cdf 1/6, 1/2, 1
             ((0.6, 0.5), (0, 1)),   # rejected -> P without x: [1/3, 2/3]
             ((0.6, 0.2), (0, 0)),
             ((0.6, 0.9), (0, 1))]
    for (u0, us), (a_want, t_want) in cases:
        U = np.array([[u0, us], [0.5, us]], np.float32)
        a, t, ma, ms = oracle.accept_stochastic(L, "f32", cu, draft, U, 1.0)
        assert (int(a[0]), int(t[0])) == (a_want, t_want), (u0, us)
        assert ma[0] >= 0.1 - 1e-7 and ms[0] > 0.05
        lo, hi = oracle.successor_interval(L, "f32", int(a[0]),
                                           2 if a_want == 0 else -1, 1.0, int(t[0]))
        assert lo <= us < hi


def test_successor_interval_exact():
    # Two rows with different logits, so a wrong row index shows.  Row 0:
    # P = [1/6, 2/6, 3/6]; row 1: P = [4/10, 1/10, 5/10] (T = 1).  Each
    # token's interval [lo, hi) in the successor distribution is the
    # cumulative probability of the tokens before it, renormalised after the
    # rejected candidate is removed.
    L = np.log(np.array([[1, 2, 3], [4, 1, 5]], np.float64)).astype(np.float32)
    sixth, tenth = 1.0 / 6.0, 0.1
    want = {
        (0, -1): [(0, sixth), (sixth, 0.5), (0.5, 1.0)],
        (0, 2): [(0, 1 / 3), (1 / 3, 1.0), (1.0, 1.0)],        # x = 2 rejected
        (0, 0): [(0, 0), (0, 0.4), (0.4, 1.0)],                # x = 0 rejected
        (0, 1): [(0, 0.25), (0.25, 0.25), (0.25, 1.0)],        # x = 1 rejected
        (1, -1): [(0, 0.4), (0.4, 0.5), (0.5, 1.0)],
        (1, 2): [(0, 0.8), (0.8, 1.0), (1.0, 1.0)],
        (1, 0): [(0, 0), (0, 1 / 6), (1 / 6, 1.0)],
        (1, 7): [(0, 0.4), (0.4, 0.5), (0.5, 1.0)],            # out-of-vocabulary id
    }
    for (row, removed), ivs in want.items():
        for tok, (lo_w, hi_w) in enumerate(ivs):
            lo, hi = oracle.successor_interval(L, "f32", row, removed, 1.0, tok)
            assert abs(lo - lo_w) < 1e-6 and abs(hi - hi_w) < 1e-6, (row, removed, tok, lo, hi)
    # temperature divides the logits: T = 2 gives P proportional to sqrt([1, 2, 3])
    r = np.sqrt([1.0, 2.0, 3.0])
    r /= r.sum()
    lo, hi = oracle.successor_interval(L, "f32", 0, -1, 2.0, 1)
    assert abs(lo - r[0]) < 1e-6 and abs(hi - r[0] - r[1]) < 1e-6
    # with x = 0 removed at T = 2
    lo, hi = oracle.successor_interval(L, "f32", 0, 0, 2.0, 2)
    assert abs(lo - r[1] / (1 - r[0])) < 1e-6 and abs(hi - 1.0) < 1e-6
    for bad in [dict(temperature=0.0), dict(token=3), dict(token=-1)]:
        kw = dict(temperature=1.0, token=0)
        kw.update(bad)
        with pytest.raises(ValueError):
            oracle.successor_interval(L, "f32", 0, -1, kw["temperature"], kw["token"])


def batch(rng, n, rows_logits, draft_block, T, dtype="f32"):
    """n identical requests of k = len(rows_logits) rows with fresh uniforms."""
    k, V = rows_logits.shape
    logits = np.tile(rows_logits, (n, 1)).astype(np.float32)
    cu = (np.arange(n + 1) * k).astype(np.int32)
    draft = np.tile(draft_block, n).astype(np.int32)
    U = rng.random((n * k, 2)).astype(np.float32)
    a, t, _, _ = oracle.accept_stochastic(logits, dtype, cu, draft, U, T)
    return a, t


@pytest.mark.parametrize("T", [0.7, 1.0, 1.6])
def test_first_emitted_token_follows_target(T):
    rng = np.random.default_rng(int(T * 100))
    V, k, n = 12, 4, 40000
    rows = rng.normal(0, 1.5, size=(k, V))
    P = softmax(rows.astype(np.float32).astype(np.float64) / T, axis=1)
    # drafts: the most likely token at each row (a deterministic top-1 drafter)
    draft_block = np.concatenate([[0], np.argmax(P[:-1], axis=1)])
    a, t = batch(rng, n, rows, draft_block, T)
    first = np.where(a >= 1, draft_block[1], t)
    counts = np.bincount(first, minlength=V)
    assert chisquare(counts, P[0] * n).pvalue > P_MIN


def test_accept_length_and_residual_distributions():
    rng = np.random.default_rng(11)
    V, k, n, T = 10, 5, 60000, 1.0
    rows = rng.normal(0, 2.0, size=(k, V))
    P = softmax(rows.astype(np.float32).astype(np.float64) / T, axis=1)
    draft_block = np.concatenate([[0], np.argmax(P[:-1], axis=1)])
    a, t = batch(rng, n, rows, draft_block, T)
    p = np.array([P[j, draft_block[j + 1]] for j in range(k - 1)])
    want = np.array([np.prod(p[:m]) * (1 - p[m]) for m in range(k - 1)] + [np.prod(p)])
    assert abs(want.sum() - 1) < 1e-12
    assert chisquare(np.bincount(a, minlength=k), want * n).pvalue > P_MIN
    # after a rejection at row 0 the successor follows P_0 without x_0
    sel = a == 0
    resid = P[0].copy()
    resid[draft_block[1]] = 0
    resid /= resid.sum()
    counts = np.bincount(t[sel], minlength=V)
    assert counts[draft_block[1]] == 0
    keep = resid > 0
    assert chisquare(counts[keep], resid[keep] * sel.sum()).pvalue > P_MIN
    # all accepted: the successor follows the last row's P unchanged
    sel = a == k - 1
    assert sel.sum() > 100
    counts = np.bincount(t[sel], minlength=V)
    assert chisquare(counts, P[k - 1] * sel.sum()).pvalue > P_MIN


def test_low_temperature_is_greedy():
    rng = np.random.default_rng(5)
    B, V = 40, 300
    k = rng.integers(1, 17, size=B)
    cu = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    cap = int(cu[-1])
    # well-separated integer logits: the argmax leads by at least 1
    logits = rng.permutation(np.tile(np.arange(V, dtype=np.float32), (cap, 1)).T).T.copy()
    logits = np.ascontiguousarray(logits)
    top = np.argmax(logits, axis=1)
    draft = rng.integers(0, V, size=cap).astype(np.int32)
    follow = rng.random(cap) < 0.7          # drafts that copy the previous row's argmax
    draft[1:][follow[1:]] = top[:-1][follow[1:]]
    U = rng.uniform(0.001, 0.999, size=(cap, 2)).astype(np.float32)
    a, t, _, _ = oracle.accept_stochastic(logits, "f32", cu, draft, U, 1e-3)
    ga, gt = oracle.accept(logits, "f32", cu, draft)
    assert np.array_equal(a, ga) and np.array_equal(t, gt)


def test_sentinels_single_rows_and_bad_ids():
    rng = np.random.default_rng(9)
    V = 50
    logits = rng.normal(size=(6, V)).astype(np.float32)
    cu = np.array([0, 0, 1, 3, 3, 6], np.int32)  # sentinel, k=1, k=2, sentinel, k=3
    draft = np.array([1, 2, -5, 4, 4, V + 3], np.int32)  # rows 2 and 5 hold invalid ids
    U = np.full((6, 2), 0.0, np.float32)   # u = 0 accepts any candidate with P > 0
    a, t, ma, ms = oracle.accept_stochastic(logits, "f32", cu, draft, U, 1.0)
    assert (a[0], t[0]) == (0, -1) and (a[3], t[3]) == (0, -1)
    assert np.isinf(ma[0]) and np.isinf(ms[3]) and np.isinf(ma[1])
    assert a[1] == 0 and t[1] == 0          # k=1: u_s = 0 draws the first token
    assert a[2] == 0                         # candidate -5 has probability 0
    assert a[4] == 1                         # candidate 4 accepted, V+3 rejected
    with pytest.raises(ValueError):
        oracle.accept_stochastic(logits, "f32", cu, draft, U, 0.0)
