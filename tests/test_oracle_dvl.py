"""Pins of the DVL allocator and packer oracle (Sec. III-C, Alg. 1,
Eqs. (6)-(11), Prop. 1).

References independent of the oracle: the paper's worked example and its
estimate-rounding example (tests/golden/paper_examples.json), scipy's expit
with numpy's running minimum for the scores, brute-force enumeration of all
length vectors on tiny batches and an exact dynamic program on larger ones
for the optimality that Prop. 1 states, and invariants of the packed layout.
"""
import itertools
import json
import os

import numpy as np
import pytest
from scipy.special import expit

import oracle
import workloads as W

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "paper_examples.json")))


def logit(p):
    return float(np.log(p / (1.0 - p)))


def objective(q, k):
    """Eq. (8): the sum over requests of their first k_i prefix scores."""
    q64 = q.astype(np.float64)
    return float(sum(q64[i, :int(k[i])].sum() for i in range(len(k))))


def seeded_rows(seeds, next_scores, w=16):
    """Logits whose scores are 1 up to position k-1, then the given score at
    position k (the next slot), then ~0; the estimate is k-1+score, so a score
    in [0.5, 1) rounds to the seed k."""
    L = np.full((len(seeds), w - 1), -40.0)
    for i, (k, v) in enumerate(zip(seeds, next_scores)):
        L[i, :k - 1] = 40.0
        if k - 1 < w - 1:
            L[i, k - 1] = logit(v)
    return L.astype(np.float32)


# ----------------------------------------------------------------- golden
def test_worked_example():
    g = GOLDEN["dvl_worked_example"]
    seeds = g["initial_lengths"]
    # R1's next slot scores highest, so the one-slot deficit grows R1
    L = seeded_rows(seeds, [0.9, 0.6, 0.55, 0.7])
    q, ell, k0 = oracle.dvl_scores(L, 16)
    assert k0.tolist() == seeds
    k, upd = oracle.dvl_adjust(q, k0, g["budget"])
    assert k.tolist() == g["lengths"] and upd == g["budget"] - sum(seeds)
    n = len(seeds)
    z = np.zeros((n, 16), np.int32)
    res = oracle.dvl_allocate_pack(L, n, z, z, z)
    assert res["k"].tolist() == g["lengths"]
    assert res["offsets"][:n].tolist() == g["offsets"]
    assert int(res["offsets"][n]) == g["end"]


def test_initial_length_rounding_example():
    g = GOLDEN["initial_length_rounding"]
    L = np.full((1, 15), -40.0)
    L[0, :6] = 40.0
    L[0, 6] = logit(0.2)
    q, ell, k0 = oracle.dvl_scores(L.astype(np.float32), 16)
    assert abs(float(ell[0]) - g["ell_hat"]) < 1e-5
    assert int(k0[0]) == g["k0"]


def test_boundary_shift_offsets():
    g = GOLDEN["boundary_shift"]
    for lengths, start in ((g["lengths_before"], g["r2_start_before"]),
                           (g["lengths_after"], g["r2_start_after"])):
        n = len(lengths)
        z = np.zeros((n, 16), np.int32)
        res = oracle.dvl_pack(np.asarray(lengths), n, 16, g["total"], z, z, z)
        assert int(res["offsets"][1]) == start
        assert int(res["offsets"][n]) == g["total"]


# ----------------------------------------------------------------- scores
def test_scores_match_expit_running_min():
    rng = np.random.default_rng(5)
    L = rng.normal(0, 3, size=(200, 15)).astype(np.float32)
    q, ell, k0 = oracle.dvl_scores(L, 16)
    ref = np.minimum.accumulate(expit(L.astype(np.float64)).astype(np.float32), axis=1)
    assert (q[:, 0] == 1.0).all()
    np.testing.assert_allclose(q[:, 1:], ref, rtol=2.4e-7, atol=0)
    assert (np.diff(q, axis=1) <= 0).all()
    np.testing.assert_allclose(ell, q[:, 1:].astype(np.float64).sum(1), rtol=1e-6)
    assert (k0 == np.clip(np.floor(ell.astype(np.float64) + 0.5), 1, 16)).all()


def test_score_special_values():
    L = np.array([[0.0, np.inf, -np.inf] + [40.0] * 12,
                  [np.inf] * 15,
                  [-np.inf] * 15,
                  [60.0] * 15], np.float32)
    q, ell, k0 = oracle.dvl_scores(L, 16)
    assert q[0, 1] == 0.5 and q[0, 2] == 0.5 and (q[0, 3:] == 0.0).all()
    assert (q[1] == 1.0).all() and ell[1] == 15.0 and k0[1] == 15
    assert (q[2, 1:] == 0.0).all() and k0[2] == 1
    assert k0[3] == 15          # the estimate never exceeds W-1
    assert k0[0] == 1           # 0.5 + 0.5 -> floor(1.0 + 0.5)


def test_scores_narrow_block():
    L = np.array([[3.0], [-3.0]], np.float32)
    q, ell, k0 = oracle.dvl_scores(L, 2)
    assert q.shape == (2, 2) and k0.tolist() == [1, 1]


# ----------------------------------------------------------------- Prop. 1
def random_case(rng, n, w, ties=False):
    raw = rng.uniform(0, 1, size=(n, w - 1))
    if ties:
        raw = np.round(raw * 4) / 4
    q = np.ones((n, w), np.float32)
    q[:, 1:] = -np.sort(-raw, axis=1)
    k0 = rng.integers(1, w + 1, size=n).astype(np.int32)
    budget = int(rng.integers(n, n * w + 1))
    return q, k0, budget


def brute_best(q, k0, budget):
    n, w = q.shape
    gap = budget - int(k0.sum())
    pref = np.concatenate([np.zeros((n, 1)), np.cumsum(q.astype(np.float64), 1)], 1)
    grids = np.array(list(itertools.product(range(1, w + 1), repeat=n)), np.int64)
    ok = grids.sum(1) == budget
    if gap > 0:
        ok &= (grids >= k0).all(1)
    elif gap < 0:
        ok &= (grids <= k0).all(1)
    else:
        ok &= (grids == k0).all(1)
    g = grids[ok]
    vals = sum(pref[i, g[:, i]] for i in range(n))
    return float(vals.max())


@pytest.mark.parametrize("n,w", [(1, 16), (2, 16), (3, 16), (4, 16), (5, 6), (6, 5)])
@pytest.mark.parametrize("ties", [False, True])
def test_prop1_optimal_against_brute_force(n, w, ties):
    rng = np.random.default_rng(100 * n + w + (7 if ties else 0))
    for _ in range(12):
        q, k0, budget = random_case(rng, n, w, ties)
        k, upd = oracle.dvl_adjust(q, k0, budget)
        gap = budget - int(k0.sum())
        assert int(k.sum()) == budget
        assert ((k >= 1) & (k <= w)).all()
        assert upd == abs(gap)
        if gap > 0:
            assert (k >= k0).all()
        elif gap < 0:
            assert (k <= k0).all()
        else:
            assert (k == k0).all()
        assert abs(objective(q, k) - brute_best(q, k0, budget)) < 1e-9


def dp_best(q, k0, budget):
    """Exact optimum of Eq. (8) under the Prop. 1 side constraints by
    dynamic programming over requests and used budget."""
    n, w = q.shape
    gap = budget - int(k0.sum())
    pref = np.concatenate([np.zeros((n, 1)), np.cumsum(q.astype(np.float64), 1)], 1)
    NEG = -np.inf
    best = np.full(budget + 1, NEG)
    best[0] = 0.0
    for i in range(n):
        lo, hi = 1, w
        if gap > 0:
            lo = int(k0[i])
        elif gap < 0:
            hi = int(k0[i])
        else:
            lo = hi = int(k0[i])
        nxt = np.full(budget + 1, NEG)
        for kk in range(lo, hi + 1):
            nxt[kk:] = np.maximum(nxt[kk:], best[:budget + 1 - kk] + pref[i, kk])
        best = nxt
    return float(best[budget])


@pytest.mark.parametrize("seed", range(4))
def test_prop1_optimal_against_dp(seed):
    rng = np.random.default_rng(40 + seed)
    d = W.make_dvl_inputs(rng, n_bs=48, n_live=48, ties=(seed % 2 == 1))
    q, ell, k0 = oracle.dvl_scores(d.pred_logits, 16)
    budget = 8 * 48
    k, upd = oracle.dvl_adjust(q, k0, budget)
    assert int(k.sum()) == budget and upd == abs(budget - int(k0.sum()))
    assert abs(objective(q, k) - dp_best(q, k0, budget)) < 1e-7


def test_zero_gap_retains_seed():
    rng = np.random.default_rng(3)
    q, k0, _ = random_case(rng, 5, 16)
    k, upd = oracle.dvl_adjust(q, k0, int(k0.sum()))
    assert (k == k0).all() and upd == 0


def test_tie_break_lowest_request_index():
    row = np.array([1.0, 0.9, 0.8, 0.8, 0.8, 0.5, 0.5, 0.2], np.float32)
    q = np.stack([row, row, row])
    k0 = np.array([3, 3, 3], np.int32)
    # growing: the next slots all score 0.8; request 0 wins, then again (its
    # next slot still scores 0.8 and it has the lowest index)
    k, _ = oracle.dvl_adjust(q, k0, 10)
    assert k.tolist() == [4, 3, 3]
    k, _ = oracle.dvl_adjust(q, k0, 11)
    assert k.tolist() == [5, 3, 3]
    # shrinking: the last slots all score 0.8; request 0 loses first
    k, _ = oracle.dvl_adjust(q, k0, 8)
    assert k.tolist() == [2, 3, 3]


def test_adjust_rejects_infeasible_budget():
    q = np.ones((2, 4), np.float32)
    with pytest.raises(ValueError):
        oracle.dvl_adjust(q, np.array([1, 1], np.int32), 9)
    with pytest.raises(ValueError):
        oracle.dvl_adjust(q, np.array([1, 1], np.int32), 1)


# ----------------------------------------------------------------- packing
@pytest.mark.parametrize("n,n_bs", [(0, 4), (1, 1), (5, 8), (32, 32)])
def test_pack_layout(n, n_bs):
    rng = np.random.default_rng(n * 31 + n_bs)
    w = 16
    d = W.make_dvl_inputs(rng, n_bs=n_bs, n_live=n)
    res = oracle.dvl_allocate_pack(d.pred_logits, n, d.tokens, d.positions, d.kv_refs, w)
    m_live, m_bs = 8 * n, 8 * n_bs
    k, off = res["k"], res["offsets"]
    assert int(k[:n].sum()) == m_live and (k[n:] == 0).all()
    assert ((k[:n] >= 1) & (k[:n] <= w)).all()
    assert off[0] == 0 and (off[n:] == m_live).all()
    assert (np.diff(off) == k).all()
    # unpacking each request's rows gives back the prefix of its block
    for i in range(n):
        s = slice(int(off[i]), int(off[i] + k[i]))
        assert (res["tokens"][s] == d.tokens[i, :k[i]]).all()
        assert (res["positions"][s] == d.positions[i, :k[i]]).all()
        assert (res["kv_refs"][s] == d.kv_refs[i, :k[i]]).all()
    # tail placeholders: token 0, position 0, the first request's first ref
    assert (res["tokens"][m_live:] == 0).all()
    assert (res["positions"][m_live:] == 0).all()
    assert (res["kv_refs"][m_live:] == d.kv_refs[0, 0]).all()
    assert res["tokens"].shape == (m_bs,)


def test_generator_gap_has_both_signs():
    gaps = []
    for s in range(12):
        d = W.make_dvl_inputs(np.random.default_rng(s), n_bs=32, n_live=32)
        _, _, k0 = oracle.dvl_scores(d.pred_logits, 16)
        gaps.append(256 - int(k0.sum()))
    assert min(gaps) < 0 < max(gaps)
