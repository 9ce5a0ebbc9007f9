"""Pins of the acceptance-predictor oracle (Sec. III-C, Eqs. (4)-(5)): the
1735-64-15 ReLU perceptron.

References independent of the oracle's matrix loops: the paper's feature and
parameter counts, explicit per-element Python loops on a tiny network,
closed forms (zero first layer, one-hot weights that select single
features, pre-activations that the ReLU must cut), and zeroed sentinel rows.
"""
import numpy as np
import pytest

import oracle
import workloads as W


def test_paper_dimensions():
    in_dim, hidden, out_dim = W.PREDICTOR_DIMS
    assert 15 * (1 + 15 + 1 + 1) == 270                 # confidence features
    assert 270 + 15 * 64 + 15 * 32 + 25 == in_dim == 1735
    assert out_dim == W.BLOCK_WIDTH - 1
    assert in_dim * hidden + hidden + hidden * out_dim + out_dim == 112079


def test_tiny_network_against_loops():
    rng = np.random.default_rng(1)
    n, i_d, h_d, o_d = 4, 5, 3, 2
    f = rng.normal(size=(n, i_d)).astype(np.float32)
    w1 = rng.normal(size=(i_d, h_d)).astype(np.float32)
    b1 = rng.normal(size=h_d).astype(np.float32)
    w2 = rng.normal(size=(h_d, o_d)).astype(np.float32)
    b2 = rng.normal(size=o_d).astype(np.float32)
    got = oracle.predictor_forward(f, n, w1, b1, w2, b2)
    for r in range(n):
        h = []
        for u in range(h_d):
            s = float(b1[u])
            for k in range(i_d):
                s += float(f[r, k]) * float(w1[k, u])
            h.append(max(s, 0.0))
        for j in range(o_d):
            s = float(b2[j])
            for u in range(h_d):
                s += h[u] * float(w2[u, j])
            assert abs(got[r, j] - s) < 1e-12


def test_closed_forms():
    rng = np.random.default_rng(2)
    d = W.make_predictor_inputs(rng, n_bs=6, n_live=6)
    in_dim, hidden, out_dim = W.PREDICTOR_DIMS
    # zero first layer: every row gives relu(b1) . W2 + b2
    z = np.zeros_like(d.w1)
    out = oracle.predictor_forward(d.features, 6, z, d.b1, d.w2, d.b2)
    want = np.maximum(d.b1.astype(np.float64), 0) @ d.w2.astype(np.float64) + d.b2
    np.testing.assert_allclose(out, np.tile(want, (6, 1)), rtol=0, atol=1e-12)
    # one-hot weights: hidden unit u reads feature 7u; output j reads unit j
    w1 = np.zeros_like(d.w1)
    w1[7 * np.arange(hidden), np.arange(hidden)] = 1.0
    w2 = np.zeros_like(d.w2)
    w2[np.arange(out_dim), np.arange(out_dim)] = 1.0
    b1 = np.zeros_like(d.b1)
    out = oracle.predictor_forward(d.features, 6, w1, b1, w2, d.b2)
    sel = d.features[:, 7 * np.arange(out_dim)].astype(np.float64)
    np.testing.assert_array_equal(out, np.maximum(sel, 0) + d.b2)
    # every pre-activation negative: the ReLU leaves only b2
    out = oracle.predictor_forward(np.abs(d.features), 6, -np.abs(d.w1), -np.abs(d.b1) - 1,
                                   d.w2, d.b2)
    np.testing.assert_array_equal(out, np.tile(d.b2.astype(np.float64), (6, 1)))


def test_sentinel_rows_are_zero():
    rng = np.random.default_rng(3)
    d = W.make_predictor_inputs(rng, n_bs=8, n_live=5)
    out = oracle.predictor_forward(d.features, 5, d.w1, d.b1, d.w2, d.b2)
    assert np.isfinite(out[:5]).all() and (out[5:] == 0).all()
    with pytest.raises(ValueError):
        oracle.predictor_forward(d.features, 9, d.w1, d.b1, d.w2, d.b2)
