"""GPU: dsv_accept_noalloc, the acceptance entry point that allocates nothing
(its chunk maxima live in the library's fixed per-device scratch), checked
bit for bit against dsv_accept with a caller workspace and against the
oracle, on calls in a row whose second input is smaller (so stale scratch
contents from the larger call must not leak into it)."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    import torch

    import paper_2609_37532_amd as dsv
    from gpu_util import AcceptDev, say
except Exception:  # pragma: no cover
    pass


def run_both(acc, name):
    """dsv_accept (workspace) and dsv_accept_noalloc on the same device
    inputs; returns both results after checking them against the oracle."""
    say("no-alloc", name, "B=%d cap=%d V=%d %s" % (acc.num_reqs, acc.capacity, acc.vocab,
                                                  acc.dtype))
    d = AcceptDev(acc)
    d.run()
    a_ws, n_ws = d.result()
    a_na = torch.full_like(d.a, -9)
    n_na = torch.full_like(d.nxt, -9)
    dsv.accept_noalloc(d.logits, d.cu, d.draft, a_na, n_na)
    torch.cuda.synchronize()
    a_na, n_na = a_na.cpu().numpy(), n_na.cpu().numpy()
    ra, rn = oracle.accept(acc.logits, acc.dtype, acc.cu_qlens, acc.draft_tokens)
    assert np.array_equal(a_na, a_ws) and np.array_equal(n_na, n_ws), name
    assert np.array_equal(a_na, ra) and np.array_equal(n_na, rn), name
    say("no-alloc", name, "ok")
    return a_na, n_na


def test_noalloc_matches_accept_on_two_calls_the_second_smaller():
    # first call: the Qwen3-8B-shaped batch (capacity 256, 151,936-token bf16
    # logits); second call: the tiny preset (capacity 32, 1,000-token fp32)
    rng = W.config_rng(4)
    attn = W.config_attn_inputs(4, rng=rng)
    big = W.config_accept_inputs(4, attn.cu_qlens, rng)
    a, n = run_both(big, "config4")
    assert np.array_equal(a, big.planted_accept_len)
    rng = W.config_rng(1)
    tiny_attn = W.config_attn_inputs(1, rng=rng)
    small = W.config_accept_inputs(1, tiny_attn.cu_qlens, rng)
    a, n = run_both(small, "config1")
    assert np.array_equal(a, small.planted_accept_len)
    assert np.array_equal(n, small.planted_next)


def test_noalloc_same_scratch_across_shapes_and_dtypes():
    # the scratch keeps the previous call's contents: a run of calls with
    # shrinking and growing shapes, both dtypes, sentinels and odd vocabularies
    rng = np.random.default_rng(4242)
    for n, (vocab, dtype, k) in enumerate([(65537, "bf16", [16, 0, 3, 9, 1]),
                                           (1001, "f32", [2, 5]),
                                           (151936, "f32", [1, 16, 16, 7, 0, 4]),
                                           (7, "bf16", [3])]):
        cu = W.cu_from_lengths(np.asarray(k, np.int32))
        acc = W.make_accept_inputs(rng, cu_qlens=cu, capacity=int(cu[-1]) + 3, vocab=vocab,
                                   dtype=dtype, p_accept=0.4)
        run_both(acc, "seq%d-V%d-%s" % (n, vocab, dtype))


def test_noalloc_rejects_a_batch_beyond_the_scratch():
    # 65,535 rows of 262,144 tokens need 16 MiB of chunk maxima: refused on
    # the host with DSV_ERR_TOO_LARGE before anything is enqueued
    lib = dsv.load()
    logits = torch.zeros((2, 8), dtype=torch.float32, device="cuda")  # never read
    i32 = lambda n: torch.zeros(n, dtype=torch.int32, device="cuda")
    rc = lib.dsv_accept_noalloc(logits.data_ptr(), 0, i32(3).data_ptr(), i32(4).data_ptr(),
                                i32(2).data_ptr(), i32(2).data_ptr(), 2, 65535, 262144, None)
    assert rc == -6
