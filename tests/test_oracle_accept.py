"""Pins of the greedy-acceptance oracle (Sec. III-D "Prefix verifier" at
temperature 0; Sec. I: accepted tokens are the contiguous candidate prefix the
target reproduces, anchor excluded; the successor comes from row offset+a).

References independent of the oracle: the planted scheme (expected results
known by construction), numpy's argmax (first occurrence wins) with a
quadratic longest-prefix search, and hand-built rows with ties.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "paper_examples.json")))


def brute_force(logits_f64, cu, draft):
    """Quadratic search: the largest m <= k-1 whose whole prefix matches."""
    B = len(cu) - 1
    a = np.zeros(B, np.int32)
    nxt = np.full(B, -1, np.int32)
    for i in range(B):
        o, k = int(cu[i]), int(cu[i + 1] - cu[i])
        if k == 0:
            continue
        t = [int(np.argmax(logits_f64[o + j])) for j in range(k)]
        best = 0
        for m in range(k - 1, -1, -1):
            if all(t[j] == draft[o + j + 1] for j in range(m)):
                best = m
                break
        a[i], nxt[i] = best, t[best]
    return a, nxt


def as_f64(inp: W.AcceptInputs):
    if inp.dtype == "f32":
        return inp.logits.astype(np.float64)
    return W.bf16_to_f32(inp.logits).astype(np.float64)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("dtype,vocab", [("f32", 1000), ("bf16", 4096)])
def test_planted_scheme(seed, dtype, vocab):
    rng = np.random.default_rng(1000 + seed)
    k = W.verify_lengths(rng, 12, 96, p=0.25)
    k[3] = 0          # a sentinel request
    k[5] = 1          # anchor only
    k[7] = 16         # full block
    cu = W.cu_from_lengths(k)
    inp = W.make_accept_inputs(rng, cu_qlens=cu, capacity=int(cu[-1]) + 5,
                               vocab=vocab, dtype=dtype, p_accept=0.3)
    a, nxt = oracle.accept(inp.logits, dtype, inp.cu_qlens, inp.draft_tokens)
    assert np.array_equal(a, inp.planted_accept_len)
    assert np.array_equal(nxt, inp.planted_next)
    ba, bn = brute_force(as_f64(inp), inp.cu_qlens, inp.draft_tokens)
    assert np.array_equal(a, ba) and np.array_equal(nxt, bn)
    assert a[3] == 0 and nxt[3] == -1
    assert a[5] == 0


def test_tiny_config_planted():
    attn = W.config_attn_inputs(1)
    rng = W.config_rng(1)
    W.config_attn_inputs(1, rng=rng)  # consume draws 1-5 in order
    inp = W.config_accept_inputs(1, attn.cu_qlens, rng)
    a, nxt = oracle.accept(inp.logits, inp.dtype, inp.cu_qlens, inp.draft_tokens)
    assert np.array_equal(a, inp.planted_accept_len)
    assert np.array_equal(nxt, inp.planted_next)
    assert (a <= np.diff(inp.cu_qlens) - 1).all()


def test_unboosted_rows_against_brute_force():
    # No planting at all: pure noise rows, random drafts that sometimes
    # match the argmax (drafts copied from the argmax for some rows).
    rng = np.random.default_rng(77)
    k = np.array([16, 4, 1, 9, 0, 16], np.int32)
    cu = W.cu_from_lengths(k)
    vocab = 257
    logits = rng.standard_normal((int(cu[-1]), vocab)).astype(np.float32)
    draft = rng.integers(0, vocab, size=int(cu[-1])).astype(np.int32)
    am = logits.astype(np.float64).argmax(axis=1)
    for r in range(len(draft) - 1):
        if rng.random() < 0.7:
            draft[r + 1] = am[r]
    a, nxt = oracle.accept(logits, "f32", cu, draft)
    ba, bn = brute_force(logits.astype(np.float64), cu, draft)
    assert np.array_equal(a, ba) and np.array_equal(nxt, bn)


def test_qlen_one_takes_anchor_row_argmax():
    rng = np.random.default_rng(3)
    cu = W.cu_from_lengths([1, 1, 1])
    logits = rng.standard_normal((3, 50)).astype(np.float32)
    draft = np.zeros(3, np.int32)
    a, nxt = oracle.accept(logits, "f32", cu, draft)
    assert (a == 0).all()
    assert np.array_equal(nxt, logits.argmax(axis=1))


def test_constant_logits_pick_index_zero():
    cu = W.cu_from_lengths([4, 2])
    logits = np.full((6, 100), 1.5, np.float32)
    draft = np.array([9, 0, 0, 5, 9, 0], np.int32)
    a, nxt = oracle.accept(logits, "f32", cu, draft)
    # request 0: drafts 0,0 then 5 -> rows 0,1 accepted (argmax 0), row 2 rejects
    assert list(a) == [2, 1] and list(nxt) == [0, 0]


def test_ties_go_to_lowest_index():
    rng = np.random.default_rng(8)
    rows, vocab = 40, 300
    x = W.bf16_bits(rng.standard_normal((rows, vocab)).astype(np.float32))
    expect = []
    for r in range(rows):
        p1, p2 = sorted(rng.choice(vocab, size=2, replace=False))
        top = W.bf16_bits(np.array([6.0], np.float32))[0]
        x[r, p2] = top
        x[r, p1] = top
        expect.append(p1)
    assert list(oracle.row_argmax(x, "bf16")) == expect


def test_signed_zero_ties():
    # -0.0 == +0.0 as values, so the lower index wins either way round.
    lg = np.full((2, 10), -1.0, np.float32)
    lg[0, 3], lg[0, 5] = 0.0, -0.0
    lg[1, 2], lg[1, 7] = -0.0, 0.0
    assert list(oracle.row_argmax(lg, "f32")) == [3, 2]
    assert list(oracle.row_argmax(W.bf16_bits(lg), "bf16")) == [3, 2]


def test_bf16_and_f32_agree_on_representable_values():
    rng = np.random.default_rng(12)
    vals = W.bf16_to_f32(W.bf16_bits(rng.standard_normal((20, 333)).astype(np.float32)))
    assert np.array_equal(oracle.row_argmax(vals, "f32"),
                          oracle.row_argmax(W.bf16_bits(vals), "bf16"))


def test_paper_worked_example_offsets():
    # Sec. III-C: lengths [6,10,7,9] pack at offsets [0,6,16,23], end 32.
    # Acceptance must read each request's rows at exactly those offsets.
    ex = GOLDEN["dvl_worked_example"]
    cu = np.array(ex["offsets"] + [ex["end"]], np.int32)
    assert np.array_equal(W.cu_from_lengths(ex["lengths"]), cu)
    rng = np.random.default_rng(21)
    inp = W.make_accept_inputs(rng, cu_qlens=cu, capacity=32, vocab=500)
    a, nxt = oracle.accept(inp.logits, "f32", cu, inp.draft_tokens)
    assert np.array_equal(a, inp.planted_accept_len)
    assert np.array_equal(nxt, inp.planted_next)


def test_rejects_bad_offsets():
    lg = np.zeros((4, 10), np.float32)
    with pytest.raises(ValueError):
        oracle.accept(lg, "f32", np.array([0, 3, 2], np.int32), np.zeros(4, np.int32))
    with pytest.raises(ValueError):
        oracle.accept(lg, "f32", np.array([0, 5], np.int32), np.zeros(4, np.int32))
