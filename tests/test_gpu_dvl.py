"""GPU parity of dsv_dvl_allocate_pack against the oracle (Sec. III-C, Alg. 1):
bit-exact scores, lengths, offsets and packed rows, through the C ABI."""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    import torch

    import paper_2609_37532_amd as dsv
    from gpu_util import DEV, DvlDev, i32_dev, say
except Exception:  # pragma: no cover
    pass

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "paper_examples.json")))
FIELDS = ("k", "offsets", "tokens", "positions", "kv_refs")


def expected(d: W.DvlInputs, n_live=None):
    n = d.n_live if n_live is None else n_live
    return oracle.dvl_allocate_pack(d.pred_logits, n, d.tokens, d.positions, d.kv_refs,
                                    d.width)


def compare(got, ref, name):
    for f in FIELDS:
        assert np.array_equal(got[f], ref[f]), (name, f, got[f], ref[f])
    gq, rq = got["q"], ref["q"]
    assert np.array_equal(gq.view(np.uint32), rq.view(np.uint32)), (name, "scores")


def check(d: W.DvlInputs, name):
    n_bs = d.tokens.shape[0]
    say("dvl", name, "n_bs=%d n_live=%d w=%d" % (n_bs, d.n_live, d.width))
    dev = DvlDev(d)
    dev.run()
    got = dev.result()
    ref = expected(d)
    compare(got, ref, name)
    say("dvl", name, "ok updates=%d" % ref["updates"])
    return got, ref


CASES = [  # (n_bs, n_live, ties, seed)
    (1, 1, False, 0), (4, 4, False, 1), (32, 32, False, 2), (32, 19, False, 3),
    (32, 32, True, 4), (64, 64, False, 5), (100, 77, True, 6), (256, 256, False, 7),
    (256, 200, True, 8), (1024, 1024, False, 9), (1024, 1024, True, 10), (1024, 1, False, 11),
    (1000, 999, False, 12), (8, 0, False, 13),
]


@pytest.mark.parametrize("n_bs,n_live,ties,seed", CASES)
def test_parity(n_bs, n_live, ties, seed):
    rng = np.random.default_rng(7000 + seed)
    d = W.make_dvl_inputs(rng, n_bs=n_bs, n_live=n_live, ties=ties)
    check(d, "n_bs%d_live%d%s" % (n_bs, n_live, "_ties" if ties else ""))


@pytest.mark.parametrize("rate_range", [(0.3, 0.6), (0.97, 0.999)])
def test_parity_large_gaps(rate_range):
    # low rates: seeds far below the budget (long grow); high rates: shrink
    rng = np.random.default_rng(7100 + int(rate_range[0] * 10))
    d = W.make_dvl_inputs(rng, n_bs=512, n_live=512, rate_range=rate_range)
    _, ref = check(d, "gap_%s" % (rate_range,))
    assert ref["updates"] > 100


@pytest.mark.parametrize("w", [2, 4, 8, 12])
def test_parity_narrow_blocks(w):
    rng = np.random.default_rng(7200 + w)
    d = W.make_dvl_inputs(rng, n_bs=96, n_live=90, width=w, ties=(w == 8))
    check(d, "w%d" % w)


def test_worked_example():
    g = GOLDEN["dvl_worked_example"]
    lg = np.full((4, 15), -40.0)
    for i, (k, v) in enumerate(zip(g["initial_lengths"], [0.9, 0.6, 0.55, 0.7])):
        lg[i, :k - 1] = 40.0
        lg[i, k - 1] = np.log(v / (1 - v))
    z = np.arange(64, dtype=np.int32).reshape(4, 16)
    d = W.DvlInputs(pred_logits=lg.astype(np.float32), n_live=4, tokens=z, positions=z + 1000,
                    kv_refs=z + 5000, width=16)
    got, _ = check(d, "worked_example")
    assert got["k"].tolist() == g["lengths"]
    assert got["offsets"].tolist() == g["offsets"] + [g["end"]]


def test_special_logits():
    rng = np.random.default_rng(7300)
    d = W.make_dvl_inputs(rng, n_bs=64, n_live=64)
    lg = d.pred_logits.copy()
    lg[0] = np.inf
    lg[1] = -np.inf
    lg[2] = 0.0
    lg[3, ::2] = np.nan
    lg[4] = -100.0          # sigmoid below the binary32 normal range
    lg[5] = 100.0
    lg[6, 3] = np.nan
    lg[7] = np.float32(1e-30)
    d.pred_logits = lg
    check(d, "special")


def test_equal_rows_tie_break():
    # every request has the same scores: the budget goes by request index
    row = np.linspace(4, -4, 15).astype(np.float32)
    for n in (3, 17, 64):
        d = W.DvlInputs(pred_logits=np.tile(row, (n, 1)), n_live=n,
                        tokens=np.zeros((n, 16), np.int32), positions=np.zeros((n, 16), np.int32),
                        kv_refs=np.zeros((n, 16), np.int32), width=16)
        check(d, "equal_rows_%d" % n)


def test_live_count_is_clamped():
    rng = np.random.default_rng(7400)
    d = W.make_dvl_inputs(rng, n_bs=48, n_live=48)
    dev = DvlDev(d)
    for raw, eff in ((-3, 0), (48 + 5, 48), (31, 31)):
        say("dvl", "clamp", raw)
        dev.num_live.fill_(raw)
        dev.run()
        compare(dev.result(), expected(d, eff), "clamp%d" % raw)


def test_without_scores_output():
    rng = np.random.default_rng(7500)
    d = W.make_dvl_inputs(rng, n_bs=32, n_live=32)
    dev = DvlDev(d)
    dev.run(scores=False)
    got = dev.result()
    ref = expected(d)
    for f in FIELDS:
        assert np.array_equal(got[f], ref[f]), f
    assert np.isnan(got["q"]).all()  # untouched


def test_graph_replay_with_changing_inputs():
    # capture once, then change the contents of the fixed buffers (live count,
    # logits, fields) between replays, as input staging does each step
    rng = np.random.default_rng(7600)
    n_bs = 64
    d0 = W.make_dvl_inputs(rng, n_bs=n_bs, n_live=n_bs)
    dev = DvlDev(d0)
    s = torch.cuda.Stream(device=DEV)
    dev.run()
    torch.cuda.synchronize()
    g = dsv.Graph().capture(lambda: dev.run(stream=s), s)
    try:
        for step, n in enumerate((64, 40, 1, 0, 63)):
            d = W.make_dvl_inputs(rng, n_bs=n_bs, n_live=n, ties=(step % 2 == 1))
            say("dvl", "graph step", step, "n", n)
            dev.logits.copy_(torch.from_numpy(d.pred_logits))
            dev.num_live.fill_(n)
            dev.tokens.copy_(torch.from_numpy(d.tokens))
            dev.positions.copy_(torch.from_numpy(d.positions))
            dev.kv_refs.copy_(torch.from_numpy(d.kv_refs))
            torch.cuda.synchronize()
            g.replay(s)
            s.synchronize()
            compare(dev.result(), expected(d), "graph%d" % step)
    finally:
        g.close()


def dvl_sweep_case(seed):
    """A seeded random bucket: size, live count, block width, tied logits and
    the acceptance-rate range (low rates make long grow loops, high rates
    long shrink loops)."""
    rng = np.random.default_rng(50_000 + seed)
    n_bs = int(rng.choice([1, 2, 3, 8, 16, 31, 32, 33, 64, 100, 255, 256, 500, 1024]))
    n_live = int(rng.integers(0, n_bs + 1)) if rng.random() < 0.5 else n_bs
    width = int(rng.choice([2, 4, 6, 8, 10, 12, 14, 16, 16, 16]))
    ties = bool(rng.random() < 0.4)
    lo = float(rng.uniform(0.2, 0.95))
    hi = float(min(0.999, lo + rng.uniform(0.01, 0.3)))
    return W.make_dvl_inputs(rng, n_bs=n_bs, n_live=n_live, width=width, ties=ties,
                             rate_range=(lo, hi))


@pytest.mark.parametrize("seed", range(24))
def test_random_sweep(seed):
    check(dvl_sweep_case(seed), "sweep%d" % seed)
