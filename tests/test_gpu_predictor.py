"""GPU parity of dsv_predictor_forward (Sec. III-C, Eq. (5), the 1735-64-15
ReLU perceptron) against the fp64 oracle, and the predictor feeding DVL.

Bound: every output must lie within the worst-case fp32 error of its
computation, derived per element from the absolute values of the terms
(recursive summation of n products with one rounding per operation stays
within gamma_n = n u / (1 - n u) of sum |terms|, u = 2^-24; the ReLU does
not enlarge an error), evaluated in float64 in the test.
"""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    import torch

    import paper_2609_37532_amd as dsv
    from gpu_util import DEV, i32_dev, say
except Exception:  # pragma: no cover
    pass

U = 2.0 ** -24


def gamma(n):
    return n * U / (1 - n * U)


def error_bound(f, n_live, w1, b1, w2, b2, ref):
    """Elementwise worst-case bound on |gpu - ref| for the live rows."""
    f64 = np.nan_to_num(f[:n_live].astype(np.float64))
    a1 = np.abs(f64) @ np.abs(w1.astype(np.float64)) + np.abs(b1.astype(np.float64))
    bh = gamma(f.shape[1] + 8) * a1                      # hidden pre-activations
    h = np.maximum(f64 @ w1.astype(np.float64) + b1, 0)
    aw2 = np.abs(w2.astype(np.float64))
    a2 = (np.abs(h) + bh) @ aw2 + np.abs(b2.astype(np.float64))
    return bh @ aw2 + gamma(w2.shape[0] + 8) * a2


class PredDev:
    def __init__(self, d: W.PredictorInputs):
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
        self.f, self.w1, self.b1, self.w2, self.b2 = (t(x) for x in
                                                      (d.features, d.w1, d.b1, d.w2, d.b2))
        self.n = i32_dev([d.n_live])
        n_bs, out_dim = d.features.shape[0], d.w2.shape[1]
        self.out = torch.full((n_bs, out_dim), float("nan"), dtype=torch.float32, device=DEV)
        self.ws = dsv.alloc_workspace(dsv.predictor_workspace_bytes(n_bs, d.features.shape[1]),
                                      DEV)

    def run(self, stream=None):
        dsv.predictor_forward(self.f, self.n, self.w1, self.b1, self.w2, self.b2, self.out,
                              workspace=self.ws, stream=stream)

    def result(self):
        torch.cuda.synchronize()
        return self.out.cpu().numpy()


def check(d: W.PredictorInputs, name):
    say("predictor", name, "n_bs", d.features.shape[0], "live", d.n_live, "dims",
        d.features.shape[1], d.w2.shape)
    dev = PredDev(d)
    dev.run()
    got = dev.result()
    ref = oracle.predictor_forward(d.features, d.n_live, d.w1, d.b1, d.w2, d.b2)
    n = d.n_live
    assert (got[n:] == 0).all(), "sentinel rows must be zero"
    assert np.isfinite(got[:n]).all()
    err = np.abs(got[:n].astype(np.float64) - ref[:n])
    bound = error_bound(d.features, n, d.w1, d.b1, d.w2, d.b2, ref)
    ratio = float((err / bound).max()) if n else 0.0
    say("predictor", name, "max err %.3g, max err/bound %.3g" % (err.max() if n else 0, ratio))
    assert (err <= bound).all()
    return got, dev


@pytest.mark.parametrize("n_bs,n_live,seed", [(1, 1, 0), (32, 32, 1), (100, 77, 2),
                                              (256, 256, 3), (1024, 1000, 4), (64, 0, 5),
                                              (8, 8, 6), (16, 11, 7), (24, 20, 8)])
def test_parity_paper_shape(n_bs, n_live, seed):
    d = W.make_predictor_inputs(np.random.default_rng(9000 + seed), n_bs=n_bs, n_live=n_live)
    check(d, "paper shape")


@pytest.mark.parametrize("dims", [(5, 64, 3), (64, 64, 15), (65, 64, 1), (4000, 64, 40),
                                  (300, 64, 100)])
def test_parity_other_shapes(dims):
    d = W.make_predictor_inputs(np.random.default_rng(9100 + dims[0]), n_bs=70, n_live=66,
                                dims=dims)
    check(d, "dims %s" % (dims,))


def test_deterministic_and_clamped():
    d = W.make_predictor_inputs(np.random.default_rng(9200), n_bs=48, n_live=48)
    got, dev = check(d, "base")
    dev.run()
    again = dev.result()
    assert np.array_equal(got.view(np.uint32), again.view(np.uint32))
    dev.n.fill_(99)    # clamped to N_bs
    dev.run()
    assert np.array_equal(dev.result().view(np.uint32), got.view(np.uint32))
    dev.n.fill_(-4)    # clamped to 0: every row zero
    dev.run()
    assert (dev.result() == 0).all()


def test_predictor_feeds_dvl_in_one_graph():
    # the decision step of Alg. 2: predictor, then DVL on its output, captured
    # once and replayed with new features each step
    rng = np.random.default_rng(9300)
    n_bs = 32
    d0 = W.make_predictor_inputs(rng, n_bs=n_bs, n_live=n_bs)
    pd = PredDev(d0)
    dv = W.make_dvl_inputs(rng, n_bs=n_bs, n_live=n_bs)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    tok, pos, ref = t(dv.tokens), t(dv.positions), t(dv.kv_refs)
    z = lambda k: torch.zeros(k, dtype=torch.int32, device=DEV)
    k, cu, pt, pp, pr = z(n_bs), z(n_bs + 1), z(8 * n_bs), z(8 * n_bs), z(8 * n_bs)
    s = torch.cuda.Stream(device=DEV)

    def decision():
        pd.run(stream=s)
        dsv.dvl_allocate_pack(pd.out, pd.n, tok, pos, ref, k, cu, pt, pp, pr, stream=s)

    decision()
    torch.cuda.synchronize()
    g = dsv.Graph().capture(decision, s)
    try:
        for step, n in enumerate((32, 20, 7, 32)):
            d = W.make_predictor_inputs(rng, n_bs=n_bs, n_live=n)
            pd.f.copy_(t(d.features))
            pd.n.fill_(n)
            torch.cuda.synchronize()
            g.replay(s)
            s.synchronize()
            logits = pd.out.cpu().numpy()
            want = oracle.predictor_forward(d.features, n, d0.w1, d0.b1, d0.w2, d0.b2)
            bound = error_bound(d.features, n, d0.w1, d0.b1, d0.w2, d0.b2, want)
            assert (np.abs(logits[:n] - want[:n]) <= bound).all()
            res = oracle.dvl_allocate_pack(logits, n, dv.tokens, dv.positions, dv.kv_refs)
            assert np.array_equal(k.cpu().numpy(), res["k"])
            assert np.array_equal(cu.cpu().numpy(), res["offsets"])
            assert np.array_equal(pt.cpu().numpy(), res["tokens"])
            say("predictor", "decision graph step", step, "live", n, "ok")
    finally:
        g.close()
