"""GPU parity of dsv_accept against the oracle: bit-exact accept lengths and
next tokens (exact argmax with lowest-index ties), through the C ABI."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    from gpu_util import AcceptDev, say
except Exception:  # pragma: no cover
    pass


def check(acc, name):
    say("accept", name, "B=%d cap=%d V=%d %s" % (acc.num_reqs, acc.capacity, acc.vocab,
                                                acc.dtype))
    d = AcceptDev(acc)
    d.run()
    a, nxt = d.result()
    ra, rn = oracle.accept(acc.logits, acc.dtype, acc.cu_qlens, acc.draft_tokens)
    assert np.array_equal(a, ra), (a, ra)
    assert np.array_equal(nxt, rn), (nxt, rn)
    say("accept", name, "ok")
    return a, nxt


def test_tiny_config():
    attn = W.config_attn_inputs(1)
    rng = W.config_rng(1)
    W.config_attn_inputs(1, rng=rng)
    acc = W.config_accept_inputs(1, attn.cu_qlens, rng)
    a, nxt = check(acc, "config1")
    assert np.array_equal(a, acc.planted_accept_len)
    assert np.array_equal(nxt, acc.planted_next)


def test_config4_shape_bf16():
    attn_rng = W.config_rng(4)
    attn = W.config_attn_inputs(4, rng=attn_rng)
    acc = W.config_accept_inputs(4, attn.cu_qlens, attn_rng)
    a, nxt = check(acc, "config4")
    assert np.array_equal(a, acc.planted_accept_len)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("vocab", [2, 7, 1000, 1001, 8192, 8193, 20011])
def test_vocab_sizes_and_alignment(dtype, vocab):
    # odd vocabularies misalign rows: exercises the scalar head/tail paths
    rng = np.random.default_rng(vocab)
    k = np.array([1, 16, 5, 0, 3], np.int32)
    cu = W.cu_from_lengths(k)
    acc = W.make_accept_inputs(rng, cu_qlens=cu, capacity=30, vocab=vocab, dtype=dtype,
                               p_accept=0.4)
    check(acc, "vocab%d-%s" % (vocab, dtype))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ties_across_chunks_and_lanes(dtype):
    rng = np.random.default_rng(4)
    vocab = 3 * 8192 + 100
    cu = W.cu_from_lengths([4, 4])
    lg = rng.standard_normal((8, vocab)).astype(np.float32)
    pairs = [(8191, 8192), (0, vocab - 1), (5, 13), (8192 * 2 + 3, 8192 * 2 + 4),
             (100, 8192 + 100), (7, 8), (1, 16385), (vocab - 2, vocab - 1)]
    for r, (p1, p2) in enumerate(pairs):
        lg[r, p1] = lg[r, p2] = 9.0
    draft = np.zeros(8, np.int32)
    logits = W.bf16_bits(lg) if dtype == "bf16" else lg
    acc = W.AcceptInputs(logits=logits, dtype=dtype, cu_qlens=cu, draft_tokens=draft,
                         planted_accept_len=np.zeros(2, np.int32),
                         planted_next=np.zeros(2, np.int32))
    a, nxt = check(acc, "ties-" + dtype)
    assert nxt[0] == pairs[0][0] and nxt[1] == pairs[4][0]


def test_signed_zero_and_constant_rows():
    cu = W.cu_from_lengths([3, 2])
    lg = np.full((5, 300), -1.0, np.float32)
    lg[0, 40], lg[0, 20] = 0.0, -0.0   # -0 at lower index wins the tie
    lg[1, :] = 2.5                     # constant row -> index 0
    lg[2, 299] = 3.0
    lg[3, 10], lg[3, 9] = -0.0, 0.0
    draft = np.array([0, 20, 0, 5, 9], np.int32)
    acc = W.AcceptInputs(logits=lg, dtype="f32", cu_qlens=cu, draft_tokens=draft,
                         planted_accept_len=np.zeros(2, np.int32),
                         planted_next=np.zeros(2, np.int32))
    a, nxt = check(acc, "signed-zero")
    assert list(a) == [2, 1] and list(nxt) == [299, 0]


def test_many_requests_random_drafts():
    rng = np.random.default_rng(8)
    k = W.verify_lengths(rng, 64, 512)
    k[::7] = 0
    cu = W.cu_from_lengths(k)
    acc = W.make_accept_inputs(rng, cu_qlens=cu, capacity=int(cu[-1]) + 9, vocab=32000,
                               dtype="bf16", p_accept=0.2)
    check(acc, "64-requests")


def test_all_sentinels():
    # no live row at all: every request still gets the sentinel outputs
    cu = np.zeros(4, np.int32)
    lg = np.zeros((6, 500), np.float32)
    acc = W.AcceptInputs(logits=lg, dtype="f32", cu_qlens=cu, draft_tokens=np.zeros(6, np.int32),
                         planted_accept_len=np.zeros(3, np.int32),
                         planted_next=np.full(3, -1, np.int32))
    a, nxt = check(acc, "all-sentinels")
    assert list(a) == [0, 0, 0] and list(nxt) == [-1, -1, -1]


def test_one_workspace_across_calls():
    # one workspace serves calls of two capacities in turn: eight calls in a
    # row, with live rows changing (none at all in one of them) and new
    # logits each time, are each exact
    import torch
    from gpu_util import DEV, bf16_dev, i32_dev
    import paper_2609_37532_amd as dsv
    B, cap, V = 12, 200, 30011
    ws = dsv.alloc_workspace(dsv.accept_workspace_bytes(cap, B, V), DEV)
    small_cap = 40  # every other call: a smaller capacity on the same workspace
    a_dev = torch.zeros(B, dtype=torch.int32, device=DEV)
    n_dev = torch.zeros(B, dtype=torch.int32, device=DEV)
    rng = np.random.default_rng(123)
    for call in range(8):
        c = cap if call % 2 == 0 else small_cap
        k = rng.integers(0, 17, size=B).astype(np.int32)
        while int(k.sum()) > c:
            k[int(np.argmax(k))] -= 1
        if call == 3:
            k[:] = 0
        cu = W.cu_from_lengths(k)
        acc = W.make_accept_inputs(rng, cu_qlens=cu, capacity=c, vocab=V, dtype="bf16",
                                   p_accept=0.35)
        say("accept", "workspace reuse", "call %d live rows %d" % (call, int(cu[-1])))
        dsv.accept(bf16_dev(acc.logits), i32_dev(cu), i32_dev(acc.draft_tokens), a_dev, n_dev,
                   workspace=ws)
        torch.cuda.synchronize()
        ra, rn = oracle.accept(acc.logits, acc.dtype, acc.cu_qlens, acc.draft_tokens)
        assert np.array_equal(a_dev.cpu().numpy(), ra), call
        assert np.array_equal(n_dev.cpu().numpy(), rn), call


def accept_sweep_case(seed):
    """A seeded random batch: request count, verify lengths with sentinels,
    capacity slack, vocabulary size (odd sizes misalign rows), dtype and the
    planted acceptance rate."""
    rng = np.random.default_rng(60_000 + seed)
    B = int(rng.choice([1, 2, 5, 16, 32, 33, 64, 200, 300]))
    k = rng.integers(0, 17, size=B).astype(np.int32)
    k[rng.random(B) < 0.1] = 0
    cu = W.cu_from_lengths(k)
    cap = int(cu[-1]) + int(rng.integers(0, 20)) + 1
    vocab = int(rng.choice([2, 3, 17, 999, 8191, 8192, 8193, 32000, 151936, 262144])
                + (rng.integers(0, 9) if rng.random() < 0.3 else 0))
    dtype = "bf16" if rng.random() < 0.6 else "f32"
    if cap * vocab > 60_000_000:
        vocab = max(2, 60_000_000 // cap)
    return W.make_accept_inputs(rng, cu_qlens=cu, capacity=cap, vocab=vocab, dtype=dtype,
                                p_accept=float(rng.uniform(0.05, 0.95)))


@pytest.mark.parametrize("seed", range(16))
def test_random_sweep(seed):
    check(accept_sweep_case(seed), "sweep%d" % seed)
