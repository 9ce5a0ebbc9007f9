"""GPU parity of dsv_verify_attn against the fp64 oracle (through the C ABI).

Bar: max-abs error <= 1e-2 (or, where the bf16 output cannot hold that,
the bf16 half-spacing at |oracle| + 2e-3, which only happens from
|oracle| = 4 up) and mean-abs error <= 1e-3 over live rows, tail rows
exactly zero, every output finite although every element the kernel must
not read is NaN (tail q rows, dead slots of last pages, spare pages).
Invariants that the design makes exact are checked bitwise (page
permutation, run-to-run determinism); packing independence and prefix
stability within one bf16 spacing of the first run's value (plus an fp32
slack of 2^-12).
"""
import zlib

import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    from gpu_util import AttnDev, assert_attn_close, assert_same_up_to_rounding, run_attn, say
except Exception:  # pragma: no cover
    pass


def oracle_out(inp):
    return oracle.verify_attn(inp.q, inp.cu_qlens, inp.kv_pages, inp.page_table,
                              inp.ctx_lens, **inp.oracle_kwargs())


def case(seed, ctx, qlens, cap=None, hq=32, hkv=8, d=128, **kw):
    rng = np.random.default_rng(seed)
    cap = cap if cap is not None else int(sum(qlens)) + 5
    return W.make_attn_inputs(rng, ctx_lens=ctx, qlens=qlens, capacity=cap,
                              num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                              spare_pages=3, **kw)


def check(inp, name, **tol):
    say("attn", name, "B=%d k=%s ctx=%s" % (inp.num_reqs, list(inp.qlens)[:8],
                                           list(inp.ctx_lens)[:8]))
    got = run_attn(inp)
    mx, mn = assert_attn_close(got, oracle_out(inp), inp, **tol)
    say("attn", name, "ok max %.3g mean %.3g" % (mx, mn))
    return got


# ------------------------------------------------------------ the presets
def test_tiny_config():
    check(W.config_attn_inputs(1), "config1-tiny")


@pytest.mark.parametrize("cfg", [2, 3])
def test_qwen_shaped_configs_all_rows(cfg):
    check(W.config_attn_inputs(cfg), "config%d" % cfg)


def test_config4_all_rows():
    check(W.config_attn_inputs(4), "config4")


# ------------------------------------------------------------ edge cases
@pytest.mark.parametrize("name,ctx,qlens", [
    ("decode-k1", [0, 1, 15, 16, 31, 32, 33, 700], [1] * 8),
    ("full-k16", [0, 5, 16, 17, 100, 511, 512, 513], [16] * 8),
    ("ragged-mix", [3, 1000, 47, 0, 2048, 9, 130, 600], [5, 1, 16, 2, 7, 13, 3, 9]),
    ("split-boundaries", [112, 113, 111, 240, 496, 497, 1008, 2032], [16, 15, 1, 16, 16, 15, 16, 16]),
])
def test_edge_lengths(name, ctx, qlens):
    check(case(zlib.crc32(name.encode()) % 1000, ctx, qlens, max_kv_len=4096), name)


def test_sentinels_and_tail():
    inp = case(5, [100, 0, 40, 0, 7], [3, 0, 16, 0, 2], cap=40)
    check(inp, "sentinels")


def test_all_sentinels_zero_every_row():
    # no live row at all: the plan has no work, every attention workgroup
    # exits at once, and the combine still zeroes all capacity rows
    inp = case(6, [300, 0, 17, 2000], [0, 0, 0, 0], cap=24)
    got = check(inp, "all-sentinels")
    assert not got.any()


def test_live_rows_fill_capacity():
    # no tail: the last request's rows end exactly at the capacity
    qlens = [16, 1, 9, 16, 4]
    check(case(8, [700, 3, 95, 1500, 64], qlens, cap=sum(qlens)), "no-tail")


@pytest.mark.parametrize("hq,hkv,d", [(4, 4, 128), (8, 4, 64), (16, 2, 128), (16, 1, 64),
                                      (32, 8, 64)])
def test_head_layouts(hq, hkv, d):
    check(case(hq * 7 + hkv + d, [300, 17, 64, 1200], [16, 4, 9, 1], hq=hq, hkv=hkv, d=d),
          "heads-%d-%d-d%d" % (hq, hkv, d))


@pytest.mark.parametrize("B", [257, 700])
def test_many_requests(B):
    # more requests than plan threads: each plan thread owns several requests
    # (and locates a share start among them); about one in six is a sentinel
    rng = np.random.default_rng(B)
    ctx = rng.integers(0, 400, size=B)
    k = rng.integers(1, 17, size=B)
    k[rng.random(B) < 0.17] = 0
    check(case(B + 11, ctx, k, hq=8, hkv=2, d=64, max_kv_len=416), "many-requests-%d" % B)


@pytest.mark.parametrize("name,ctx,qlens", [
    # one long request: the small-batch plan cuts its 8 segments into about
    # 30 pieces each (a piece cap above 8 blocks to stay within one per CU),
    # so the combine merges far more than 8 partials per row
    ("one-long-request", [8000], [16]),
    ("two-requests-one-long", [7000, 40], [9, 16]),
])
def test_small_batch_many_pieces(name, ctx, qlens):
    check(case(zlib.crc32(name.encode()) % 1000, ctx, qlens, max_kv_len=8016), name)


def test_large_outputs_bf16_bound():
    # Many very short contexts at G = 16: with a handful of keys an output
    # reaches |x| > 4, where rounding to bf16 alone moves it by up to 0.0156.
    # The flat 1e-2 is then out of reach for any bf16 output (the oracle's
    # own bf16 rounding breaks it here); the bound takes the format into
    # account there and stays 1e-2 below |x| ~ 2.
    import torch
    from gpu_util import attn_bound
    c = sweep_case(111)
    inp = case(c["seed"], c["ctx"], c["qlens"], cap=c["cap"], hq=c["hq"], hkv=c["hkv"],
               d=c["d"], max_kv_len=max(c["max_kv_len"], 1))
    ref = oracle_out(inp)
    live = int(inp.cu_qlens[-1])
    r = ref[:live]
    rounded = torch.from_numpy(r.astype(np.float32)).to(torch.bfloat16).double().numpy()
    assert np.abs(rounded - r).max() > 1e-2  # the flat bound is unattainable here
    assert (np.abs(rounded - r) <= attn_bound(r)).all()  # the format-aware one is not
    check(inp, "large-outputs")


def test_long_context():
    check(case(77, [16000, 9000, 31], [4, 16, 2], max_kv_len=16384), "long-context")


def test_peaked_scores():
    # Q scaled by 4 makes the softmax peaky: few keys carry the weight, so
    # the bf16 rounding of the weights averages out less.  Every element is
    # still held to the per-element bound (1e-2 below |x| = 4); the mean is
    # reported, not bounded, since it is no longer an average over many
    # small independent errors.
    from gpu_util import attn_bound
    inp = case(91, [800, 50, 2000, 9], [16, 3, 6, 1], q_scale=4.0)
    say("attn", "peaked")
    got = run_attn(inp)
    ref = oracle_out(inp)
    live = int(inp.cu_qlens[-1])
    assert np.isfinite(got).all()
    err = np.abs(got[:live] - ref[:live])
    say("attn", "peaked: max %.3g mean %.3g" % (err.max(), err.mean()))
    assert (err <= attn_bound(ref[:live])).all(), float(err.max())


def test_closed_form_single_key_is_exact():
    # ctx = 0, k = 1: one key with weight 1 -> out == V_0 exactly (bf16).
    inp = case(13, [0, 0, 0], [1, 1, 1])
    say("attn", "single-key")
    got = run_attn(inp)
    ref = oracle_out(inp)
    live = int(inp.cu_qlens[-1])
    assert np.array_equal(got[:live], ref[:live])


# ------------------------------------------------------------ exact invariants
def test_packing_independence():
    # The same requests packed in another order, with sentinels and another
    # capacity, give the same rows up to rounding: the stream-K share
    # boundaries depend on the batch's total work, so another packing can
    # cut a request's segments elsewhere, which changes its fp32 summation
    # order (weights only move by powers of two).
    inp = W.config_attn_inputs(3)
    say("attn", "packing independence")
    base = run_attn(inp)
    B = inp.num_reqs
    rng = np.random.default_rng(3)
    for trial in range(2):
        order = list(rng.permutation(B))
        gaps = list(rng.integers(0, 2, size=B + 1))
        alt = W.repack(inp, order, capacity=int(inp.qlens.sum()) + 17, gaps=gaps)
        got = run_attn(alt)
        worst = 0.0
        for old_i, new_i, o_old, o_new, k in alt.meta["moves"]:
            worst = max(worst, assert_same_up_to_rounding(
                got[o_new:o_new + k], base[o_old:o_old + k], "request %d" % old_i))
        say("attn", "packing trial %d: max diff %.3g" % (trial, worst))
        assert not got[int(alt.cu_qlens[-1]):].any()


def test_page_permutation_bitwise():
    inp = case(29, [900, 41, 3000], [8, 3, 16])
    say("attn", "page permutation")
    base = run_attn(inp)
    perm = np.random.default_rng(5).permutation(inp.num_pages)
    kv2 = np.empty_like(inp.kv_pages)
    kv2[perm] = inp.kv_pages
    pt2 = np.where(inp.page_table >= 0, perm[np.maximum(inp.page_table, 0)], -1)
    alt = W.AttnInputs(q=inp.q, cu_qlens=inp.cu_qlens, kv_pages=kv2,
                       page_table=pt2.astype(np.int32), ctx_lens=inp.ctx_lens,
                       num_q_heads=inp.num_q_heads, num_kv_heads=inp.num_kv_heads,
                       head_dim=inp.head_dim, page_size=inp.page_size,
                       max_kv_len=inp.max_kv_len, scale=inp.scale)
    assert np.array_equal(run_attn(alt), base)


def test_determinism_bitwise():
    inp = W.config_attn_inputs(4)
    say("attn", "determinism x20")
    d = AttnDev(inp)
    d.run()
    first = d.result()
    for _ in range(20):
        d.run()
    assert np.array_equal(d.result(), first)


def test_prefix_stability_up_to_rounding():
    # Row j does not depend on k_i while j < k_i, up to rounding: the work
    # split and the rows that share a tile change with the number of live
    # rows.
    base = case(31, [1500], [16], cap=16)
    say("attn", "prefix stability")
    full = run_attn(base)
    for k in (1, 3, 4, 5, 8, 13):
        alt = W.AttnInputs(q=base.q, cu_qlens=np.array([0, k], np.int32),
                           kv_pages=base.kv_pages, page_table=base.page_table,
                           ctx_lens=base.ctx_lens, num_q_heads=base.num_q_heads,
                           num_kv_heads=base.num_kv_heads, head_dim=base.head_dim,
                           page_size=base.page_size, max_kv_len=base.max_kv_len,
                           scale=base.scale)
        got = run_attn(alt)
        d = assert_same_up_to_rounding(got[:k], full[:k], "k=%d" % k)
        say("attn", "prefix stability k=%d: max diff %.3g" % (k, d))


# ------------------------------------------------------------ random sweep
def sweep_case(seed):
    """A seeded random batch: head layout, batch size, context distribution,
    verify lengths (with sentinels), capacity slack.  Contexts are redrawn
    shorter until the oracle's work stays near a second.  The kind cycles
    with the seed so both plans are reached: small batches cut whole
    segments into pieces, and the last kind (many KV heads, few query rows,
    long contexts) always takes stream-K shares that straddle segments."""
    rng = np.random.default_rng(10_000 + seed)
    kind = seed % 5
    G = int(rng.choice([1, 2, 4, 8, 16]))
    hkv = int(rng.choice([1, 2, 4, 8]))
    while G * hkv > 64:
        hkv //= 2
    d = int(rng.choice([64, 128]))
    B = int(rng.choice([1, 2, 3, 5, 8, 13, 24, 40, 96, 300]))
    kmax = 17
    if kind == 4:
        G, hkv, d = int(rng.choice([1, 2])), 8, 64
        B, kmax = int(rng.choice([24, 40, 96])), 5
    k = rng.integers(1, kmax, size=B)
    k[rng.random(B) < 0.15] = 0
    hi = 4000
    while True:
        if kind == 0:    # uniform
            ctx = rng.integers(0, hi, size=B)
        elif kind == 1:  # ctx + k on or next to 32-key block edges
            ctx = np.maximum(0, 32 * rng.integers(0, hi // 32, size=B) - k
                             + rng.integers(-1, 2, size=B))
        elif kind == 2:  # one long request among short ones
            ctx = rng.integers(0, 64, size=B)
            ctx[int(rng.integers(0, B))] = int(rng.integers(hi // 2, hi))
        elif kind == 3:  # short contexts only
            ctx = rng.integers(0, 48, size=B)
        else:            # long contexts
            ctx = rng.integers(hi // 4, hi, size=B)
        work = float(np.sum(k.astype(np.float64) * G * hkv * (ctx + k) * d))
        if work <= 4e8 or hi <= 64:
            break
        hi //= 2
    cap = int(k.sum()) + int(rng.integers(0, 24))
    return dict(seed=seed, ctx=ctx, qlens=k, cap=max(cap, 1), hq=G * hkv, hkv=hkv, d=d,
                max_kv_len=int((ctx + k).max()) + int(rng.integers(0, 40)))


@pytest.mark.parametrize("seed", range(32))
def test_random_sweep(seed):
    c = sweep_case(seed)
    check(case(c["seed"], c["ctx"], c["qlens"], cap=c["cap"], hq=c["hq"], hkv=c["hkv"],
               d=c["d"], max_kv_len=max(c["max_kv_len"], 1)),
          "sweep-%d hq=%d hkv=%d d=%d" % (seed, c["hq"], c["hkv"], c["d"]))
