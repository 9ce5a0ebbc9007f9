"""GPU parity of dsv_accept_stochastic (Sec. III-D prefix verifier, T > 0)
through the C ABI.

The result is a function of the caller's uniforms, so each request is
compared exactly with the fp64 oracle unless one of its uniforms lies within
TOL = 1e-5 of the threshold it was compared with (the oracle reports that
margin); such requests only have to be valid, and the successor must occupy
a cumulative interval within TOL of its uniform.  Independently of the oracle, a
chi-square test checks that the first token the GPU emits follows the target
distribution of the anchor row (the verifier is lossless), and at very low
temperature the result must equal the greedy verifier's.
"""
import numpy as np
import pytest
from scipy.special import softmax
from scipy.stats import chisquare

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    import torch

    import paper_2609_37532_amd as dsv
    from gpu_util import DEV, bf16_dev, i32_dev, say
except Exception:  # pragma: no cover
    pass

TOL = 1e-5  # in probability: accept thresholds and cumulative positions


def make_case(rng, B, V, dtype, kmax=16, p_follow=0.8, sentinels=True):
    """Random lengths (with sentinels and k=1), N(0,1) logits, and drafts
    whose logit gets a boost so that candidates carry real probability."""
    k = rng.integers(1, kmax + 1, size=B)
    if sentinels and B > 3:
        k[1] = 0
        k[2] = 1
    cu = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    cap = int(cu[-1]) + 3
    logits = rng.standard_normal((cap, V), dtype=np.float32)
    draft = rng.integers(0, V, size=cap).astype(np.int32)
    boost_hi = float(np.log(V)) + 4.0
    for i in range(B):
        o = int(cu[i])
        for j in range(int(k[i]) - 1):
            if rng.random() < p_follow:
                logits[o + j, draft[o + j + 1]] += rng.uniform(boost_hi - 6.0, boost_hi)
    U = rng.random((cap, 2)).astype(np.float32)
    if dtype == "bf16":
        logits = W.bf16_bits(logits)
    return logits, cu, draft, U


def run_gpu(logits, dtype, cu, draft, U, T):
    lg = bf16_dev(logits) if dtype == "bf16" else torch.from_numpy(logits).to(DEV)
    B = cu.shape[0] - 1
    a = torch.full((B,), -7, dtype=torch.int32, device=DEV)
    nxt = torch.full((B,), -7, dtype=torch.int32, device=DEV)
    dsv.accept_stochastic(lg, i32_dev(cu), i32_dev(draft), torch.from_numpy(U).to(DEV), T, a,
                          nxt)
    torch.cuda.synchronize()
    return a.cpu().numpy(), nxt.cpu().numpy()


def compare(ga, gt, logits, dtype, cu, draft, U, T, name):
    """Per live request: the accepted length equals the oracle's unless an
    accept-test uniform lies within TOL of its threshold; the successor
    (drawn under the GPU's accepted length) occupies, in the oracle's
    cumulative distribution, an interval of positive probability within TOL
    of the successor uniform, and equals the oracle's token when both
    margins exceed TOL."""
    ra, rt, ma, ms = oracle.accept_stochastic(logits, dtype, cu, draft, U, T)
    B, V = cu.shape[0] - 1, logits.shape[1]
    exact_a = exact_t = 0
    for i in range(B):
        o, k = int(cu[i]), int(cu[i + 1] - cu[i])
        if k == 0:
            assert (ga[i], gt[i]) == (0, -1)
            continue
        a = int(ga[i])
        assert 0 <= a <= k - 1, (name, i, a)
        if ma[i] > TOL:
            assert a == ra[i], (name, i, a, ra[i], ma[i])
            exact_a += 1
        r = o + a
        x = int(draft[r + 1]) if a < k - 1 else -1
        removed = x if 0 <= x < V else -1
        t = int(gt[i])
        assert 0 <= t < V and t != removed, (name, i, t)
        lo, hi = oracle.successor_interval(logits, dtype, r, removed, T, t)
        u = float(U[r, 1])
        assert hi > lo and lo - TOL <= u < hi + TOL, (name, i, t, lo, hi, u)
        if a == ra[i] and ma[i] > TOL and ms[i] > TOL:
            assert t == rt[i], (name, i, t, rt[i])
            exact_t += 1
    live = np.diff(cu) > 0
    say("sample", name, "live %d, accept exact %d, successor exact %d, mean accepted %.2f"
        % (int(live.sum()), exact_a, exact_t, float(ga[live].mean())))


@pytest.mark.parametrize("dtype,V,B,T,seed", [
    ("f32", 1000, 24, 1.0, 0), ("f32", 1000, 24, 0.5, 1), ("f32", 300, 40, 2.0, 2),
    ("bf16", 10007, 16, 1.0, 3), ("bf16", 16384, 8, 0.7, 4), ("f32", 8193, 12, 1.3, 5),
    ("bf16", 151936, 32, 1.0, 6),
])
def test_parity(dtype, V, B, T, seed):
    rng = np.random.default_rng(8000 + seed)
    logits, cu, draft, U = make_case(rng, B, V, dtype)
    ga, gt = run_gpu(logits, dtype, cu, draft, U, T)
    compare(ga, gt, logits, dtype, cu, draft, U, T, "%s V=%d B=%d T=%g" % (dtype, V, B, T))


def test_first_emitted_token_follows_target():
    rng = np.random.default_rng(8100)
    V, k, n, T = 12, 4, 16000, 0.9  # capacity n*k stays within 65535 rows
    rows = rng.normal(0, 1.5, size=(k, V)).astype(np.float32)
    P = softmax(rows.astype(np.float64) / T, axis=1)
    draft_block = np.concatenate([[0], np.argmax(P[:-1], axis=1)]).astype(np.int32)
    logits = np.tile(rows, (n, 1))
    cu = (np.arange(n + 1) * k).astype(np.int32)
    draft = np.tile(draft_block, n)
    U = rng.random((n * k, 2)).astype(np.float32)
    a, t = run_gpu(logits, "f32", cu, draft, U, T)
    first = np.where(a >= 1, draft_block[1], t)
    counts = np.bincount(first, minlength=V)
    say("sample", "chi-square first token", counts.tolist())
    assert chisquare(counts, P[0] * n).pvalue > 1e-4
    p = np.array([P[j, draft_block[j + 1]] for j in range(k - 1)])
    want = np.array([np.prod(p[:m]) * (1 - p[m]) for m in range(k - 1)] + [np.prod(p)])
    assert chisquare(np.bincount(a, minlength=k), want * n).pvalue > 1e-4


def test_low_temperature_equals_greedy():
    rng = np.random.default_rng(8200)
    B, V = 32, 4096
    k = rng.integers(1, 17, size=B)
    cu = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    cap = int(cu[-1])
    logits = np.stack([rng.permutation(V) for _ in range(cap)]).astype(np.float32)
    top = np.argmax(logits, axis=1)
    draft = rng.integers(0, V, size=cap).astype(np.int32)
    follow = rng.random(cap) < 0.8
    draft[1:][follow[1:]] = top[:-1][follow[1:]]
    U = rng.uniform(0.001, 0.999, size=(cap, 2)).astype(np.float32)
    a, t = run_gpu(logits, "f32", cu, draft, U, 1e-3)
    ga, gt = oracle.accept(logits, "f32", cu, draft)
    bad = np.nonzero((a != ga) | (t != gt))[0]
    for i in bad[:6]:
        o = int(cu[i])
        say("sample", "low T mismatch req", int(i), "k", int(k[i]), "gpu", int(a[i]), int(t[i]),
            "greedy", int(ga[i]), int(gt[i]), "draft==top", [bool(draft[o + j + 1] == top[o + j])
                                                            for j in range(int(k[i]) - 1)])
    assert bad.size == 0


def test_masked_vocabulary_and_bad_ids():
    rng = np.random.default_rng(8300)
    logits, cu, draft, U = make_case(rng, 20, 5000, "f32")
    logits[:, 1::2] = -np.inf                # odd tokens are banned
    draft[5] = -3
    draft[9] = 5000 + 11
    T = 1.0
    ga, gt = run_gpu(logits, "f32", cu, draft, U, T)
    compare(ga, gt, logits, "f32", cu, draft, U, T, "masked")
    live = np.diff(cu) > 0
    assert (gt[live] % 2 == 0).all()


def test_graph_replay_with_changing_uniforms():
    rng = np.random.default_rng(8400)
    logits, cu, draft, U = make_case(rng, 16, 20000, "bf16")
    T = 0.8
    lg = bf16_dev(logits)
    B = cu.shape[0] - 1
    cu_d, dr_d = i32_dev(cu), i32_dev(draft)
    u_d = torch.from_numpy(U).to(DEV)
    a = torch.zeros(B, dtype=torch.int32, device=DEV)
    nxt = torch.zeros(B, dtype=torch.int32, device=DEV)
    ws = dsv.alloc_workspace(dsv.accept_stochastic_workspace_bytes(lg.shape[0], B, 20000), DEV)
    s = torch.cuda.Stream(device=DEV)
    fn = lambda: dsv.accept_stochastic(lg, cu_d, dr_d, u_d, T, a, nxt, workspace=ws, stream=s)
    fn()
    torch.cuda.synchronize()
    g = dsv.Graph().capture(fn, s)
    try:
        for rep in range(4):
            U = rng.random(U.shape).astype(np.float32)
            u_d.copy_(torch.from_numpy(U))
            torch.cuda.synchronize()
            g.replay(s)
            s.synchronize()
            compare(a.cpu().numpy(), nxt.cpu().numpy(), logits, "bf16", cu, draft, U, T,
                    "graph replay %d" % rep)
    finally:
        g.close()
