"""Pins of the fp64 attention oracle against things other than itself.

Each check targets a plausible oracle mistake: a wrong causal offset, a wrong
GQA head map, a wrong scale, a mis-decoded page layout, reading the wrong
packed row, or touching memory it must not read (NaN poison).  References:
  - dense brute force: gather the request's keys into dense [L, Hkv, D]
    arrays through the page table and run masked softmax attention as whole
    matrices (numpy, float64);
  - a library routine: torch's scaled_dot_product_attention in float64 on
    the CPU with an explicit boolean mask (square causal case: is_causal);
  - closed forms and invariants of the definition (Sec. III-D, Eq. (16)).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "paper_examples.json")))


def dense_kv(inp: W.AttnInputs, i: int):
    """Request i's logical K, V as float64 [L, Hkv, D] (test-side decoding)."""
    L = int(inp.ctx_lens[i] + inp.qlens[i])
    ps, D, Hkv = inp.page_size, inp.head_dim, inp.num_kv_heads
    t = np.arange(L)
    page = inp.page_table[i, t // ps]
    slot = t % ps
    d = np.arange(D)
    heads = np.arange(Hkv)
    koff = W.k_tile_offset(slot[:, None], d[None, :], ps)
    voff = W.v_tile_offset(slot[:, None], d[None, :], ps)
    K = inp.kv_pages[page[:, None, None], 0, heads[None, :, None], koff[:, None, :]]
    V = inp.kv_pages[page[:, None, None], 1, heads[None, :, None], voff[:, None, :]]
    return (W.bf16_to_f32(K).astype(np.float64), W.bf16_to_f32(V).astype(np.float64))


def brute_force(inp: W.AttnInputs) -> np.ndarray:
    """Masked softmax attention as whole matrices, one request at a time."""
    out = np.zeros((inp.capacity, inp.num_q_heads, inp.head_dim))
    G = inp.num_q_heads // inp.num_kv_heads
    for i in range(inp.num_reqs):
        o, k, ctx = int(inp.cu_qlens[i]), int(inp.qlens[i]), int(inp.ctx_lens[i])
        if k == 0:
            continue
        K, V = dense_kv(inp, i)
        L = ctx + k
        allowed = np.arange(L)[None, :] <= (ctx + np.arange(k))[:, None]
        for h in range(inp.num_q_heads):
            Q = W.bf16_to_f32(inp.q[o:o + k, h]).astype(np.float64)
            S = inp.scale * (Q @ K[:, h // G].T)
            S = np.where(allowed, S, -np.inf)
            P = np.exp(S - S.max(axis=1, keepdims=True))
            out[o:o + k, h] = (P @ V[:, h // G]) / P.sum(axis=1, keepdims=True)
    return out


def sdpa_reference(inp: W.AttnInputs) -> np.ndarray:
    """torch SDPA (float64, CPU) with an explicit boolean mask per request."""
    out = np.zeros((inp.capacity, inp.num_q_heads, inp.head_dim))
    G = inp.num_q_heads // inp.num_kv_heads
    for i in range(inp.num_reqs):
        o, k, ctx = int(inp.cu_qlens[i]), int(inp.qlens[i]), int(inp.ctx_lens[i])
        if k == 0:
            continue
        K, V = dense_kv(inp, i)
        L = ctx + k
        q = torch.from_numpy(W.bf16_to_f32(inp.q[o:o + k]).astype(np.float64))
        q = q.permute(1, 0, 2).unsqueeze(0)                          # [1,Hq,k,D]
        kt = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(G, 0)[None]
        vt = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(G, 0)[None]
        mask = torch.arange(L)[None, :] <= (ctx + torch.arange(k))[:, None]
        r = torch.nn.functional.scaled_dot_product_attention(
            q, kt, vt, attn_mask=mask, scale=inp.scale)
        out[o:o + k] = r[0].permute(1, 0, 2).numpy()
    return out


def run_oracle(inp: W.AttnInputs) -> np.ndarray:
    return oracle.verify_attn(inp.q, inp.cu_qlens, inp.kv_pages, inp.page_table,
                              inp.ctx_lens, **inp.oracle_kwargs())


def small_case(seed, ctx, qlens, cap=None, hq=8, hkv=2, d=64, **kw):
    rng = np.random.default_rng(seed)
    cap = cap if cap is not None else int(sum(qlens)) + 3
    return W.make_attn_inputs(rng, ctx_lens=ctx, qlens=qlens, capacity=cap,
                              num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                              spare_pages=2, **kw)


# ---------------------------------------------------------------- brute force
def test_tiny_config_matches_brute_force_and_sdpa():
    inp = W.config_attn_inputs(1)
    got = run_oracle(inp)
    assert np.isfinite(got).all()
    np.testing.assert_allclose(got, brute_force(inp), rtol=0, atol=1e-12)
    np.testing.assert_allclose(got, sdpa_reference(inp), rtol=0, atol=1e-12)


@pytest.mark.parametrize("hq,hkv", [(8, 2), (8, 8), (16, 1), (6, 3)])
def test_gqa_groups_match_sdpa(hq, hkv):
    # Hkv > 1 pins the head -> KV-head map (h // G, not h % Hkv).
    inp = small_case(7 + hq + hkv, ctx=[0, 17, 33, 64], qlens=[3, 16, 1, 9],
                     hq=hq, hkv=hkv)
    np.testing.assert_allclose(run_oracle(inp), sdpa_reference(inp), rtol=0,
                               atol=1e-12)


def test_head_dim_128_and_custom_scale():
    inp = small_case(11, ctx=[40, 5], qlens=[7, 12], d=128, scale=0.3)
    np.testing.assert_allclose(run_oracle(inp), brute_force(inp), rtol=0, atol=1e-12)


# --------------------------------------------------------------- closed forms
def test_single_key_returns_v0_exactly():
    # ctx = 0, k = 1: one visible key, weight exactly 1 -> out == V_0.
    inp = small_case(3, ctx=[0, 0], qlens=[1, 1])
    got = run_oracle(inp)
    G = inp.num_q_heads // inp.num_kv_heads
    for i in range(2):
        _, V = dense_kv(inp, i)
        for h in range(inp.num_q_heads):
            assert np.array_equal(got[inp.cu_qlens[i], h], V[0, h // G])


def test_constant_v_gives_constant():
    inp = small_case(5, ctx=[30, 3], qlens=[5, 16])
    c = W.bf16_bits(np.float32(0.8125))
    inp.kv_pages[:, 1] = c  # every V element; the layout is irrelevant here
    got = run_oracle(inp)
    live = int(inp.cu_qlens[-1])
    np.testing.assert_allclose(got[:live], 0.8125, rtol=0, atol=1e-14)


def test_zero_keys_give_mean_of_visible_values():
    inp = small_case(9, ctx=[21, 0], qlens=[4, 6])
    inp.kv_pages[:, 0] = 0  # K == 0: all scores equal, uniform weights
    got = run_oracle(inp)
    G = inp.num_q_heads // inp.num_kv_heads
    for i in range(2):
        _, V = dense_kv(inp, i)
        o, ctx = int(inp.cu_qlens[i]), int(inp.ctx_lens[i])
        for j in range(int(inp.qlens[i])):
            mean = V[:ctx + j + 1].mean(axis=0)  # [Hkv, D]
            for h in range(inp.num_q_heads):
                np.testing.assert_allclose(got[o + j, h], mean[h // G], atol=1e-13)


# ----------------------------------------------------------------- invariants
def test_qlen_one_is_decode_attention():
    # k = 1: ordinary decode attention of one query over ctx + 1 keys.
    inp = small_case(13, ctx=[50, 77, 0], qlens=[1, 1, 1])
    got = run_oracle(inp)
    G = inp.num_q_heads // inp.num_kv_heads
    for i in range(3):
        K, V = dense_kv(inp, i)
        o = int(inp.cu_qlens[i])
        for h in range(inp.num_q_heads):
            q = torch.from_numpy(W.bf16_to_f32(inp.q[o, h]).astype(np.float64))
            r = torch.nn.functional.scaled_dot_product_attention(
                q[None, None, None], torch.from_numpy(K[:, h // G])[None, None],
                torch.from_numpy(V[:, h // G])[None, None], scale=inp.scale)
            np.testing.assert_allclose(got[o, h], r.numpy()[0, 0, 0], atol=1e-12)


def test_full_block_is_last_rows_of_causal_attention():
    # k = 16: the block rows equal the last 16 rows of ordinary (square)
    # causal attention over ctx + 16 positions.
    ctx = 45
    inp = small_case(17, ctx=[ctx], qlens=[16], hq=4, hkv=1)
    got = run_oracle(inp)
    K, V = dense_kv(inp, 0)
    L = ctx + 16
    rng = np.random.default_rng(99)
    qfull = rng.standard_normal((L, 4, inp.head_dim))
    qfull[ctx:] = W.bf16_to_f32(inp.q[:16]).astype(np.float64)
    r = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(qfull).permute(1, 0, 2)[None],
        torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(4, 0)[None],
        torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(4, 0)[None],
        is_causal=True, scale=inp.scale)
    np.testing.assert_allclose(got[:16], r[0].permute(1, 0, 2).numpy()[ctx:],
                               atol=1e-12)


def test_packing_independence_is_exact():
    inp = small_case(19, ctx=[10, 60, 33, 5], qlens=[6, 10, 7, 9], cap=40)
    ref = run_oracle(inp)
    # paper worked example of the packer: these lengths at these offsets
    ex = GOLDEN["dvl_worked_example"]
    assert list(inp.qlens) == ex["lengths"]
    assert list(inp.cu_qlens) == ex["offsets"] + [ex["end"]]
    for order, gaps, cap in [([3, 1, 0, 2], [1, 0, 2, 0, 1], 50),
                             ([2, 0, 3, 1], None, 32),
                             ([0, 1, 2, 3], [0, 0, 0, 0, 3], 64)]:
        alt = W.repack(inp, order, capacity=cap, gaps=gaps)
        got = run_oracle(alt)
        for old_i, new_i, o_old, o_new, k in alt.meta["moves"]:
            assert np.array_equal(got[o_new:o_new + k], ref[o_old:o_old + k])
        assert not got[int(alt.cu_qlens[-1]):].any()


def test_paper_boundary_shift_keeps_each_requests_rows():
    # Sec. II-C: lengths [4,12,8] -> [10,8,6]; R2's rows move from offset 4 to
    # 10.  With the same request data, every row present in both steps is
    # identical (packing independence + prefix stability).
    ex = GOLDEN["boundary_shift"]
    before, after = ex["lengths_before"], ex["lengths_after"]
    ctx = [31, 8, 70]
    full = small_case(23, ctx=ctx, qlens=[16, 16, 16], cap=48)
    full_out = run_oracle(full)

    def step(lengths):
        q = np.full((24, full.num_q_heads, full.head_dim), W.BF16_NAN, np.uint16)
        cu = W.cu_from_lengths(lengths)
        for i, k in enumerate(lengths):
            q[cu[i]:cu[i] + k] = full.q[16 * i:16 * i + k]
        s = W.AttnInputs(q=q, cu_qlens=cu, kv_pages=full.kv_pages,
                         page_table=full.page_table, ctx_lens=full.ctx_lens,
                         num_q_heads=full.num_q_heads,
                         num_kv_heads=full.num_kv_heads, head_dim=full.head_dim,
                         page_size=full.page_size, max_kv_len=full.max_kv_len,
                         scale=full.scale)
        return cu, run_oracle(s)

    cu_b, out_b = step(before)
    cu_a, out_a = step(after)
    assert int(cu_b[1]) == ex["r2_start_before"] and int(cu_a[1]) == ex["r2_start_after"]
    assert int(cu_b[-1]) == int(cu_a[-1]) == ex["total"]
    for i in range(3):
        m = min(before[i], after[i])
        assert np.array_equal(out_b[cu_b[i]:cu_b[i] + m], out_a[cu_a[i]:cu_a[i] + m])
        assert np.array_equal(out_b[cu_b[i]:cu_b[i] + m], full_out[16 * i:16 * i + m])


def test_page_permutation_invariance_is_exact():
    inp = small_case(29, ctx=[90, 41], qlens=[8, 3])
    ref = run_oracle(inp)
    rng = np.random.default_rng(5)
    perm = rng.permutation(inp.num_pages)          # old id -> new id
    kv2 = np.empty_like(inp.kv_pages)
    kv2[perm] = inp.kv_pages
    pt2 = np.where(inp.page_table >= 0, perm[np.maximum(inp.page_table, 0)], -1)
    alt = W.AttnInputs(q=inp.q, cu_qlens=inp.cu_qlens, kv_pages=kv2,
                       page_table=pt2.astype(np.int32), ctx_lens=inp.ctx_lens,
                       num_q_heads=inp.num_q_heads, num_kv_heads=inp.num_kv_heads,
                       head_dim=inp.head_dim, page_size=inp.page_size,
                       max_kv_len=inp.max_kv_len, scale=inp.scale)
    assert np.array_equal(run_oracle(alt), ref)


def test_prefix_stability():
    # Row j does not depend on k_i while j < k_i (causality inside the block).
    base = small_case(31, ctx=[52], qlens=[16])
    ref = run_oracle(base)
    for k in (1, 5, 11):
        cu = np.array([0, k], np.int32)
        alt = W.AttnInputs(q=base.q, cu_qlens=cu, kv_pages=base.kv_pages,
                           page_table=base.page_table, ctx_lens=base.ctx_lens,
                           num_q_heads=base.num_q_heads,
                           num_kv_heads=base.num_kv_heads, head_dim=base.head_dim,
                           page_size=base.page_size, max_kv_len=base.max_kv_len,
                           scale=base.scale)
        assert np.array_equal(run_oracle(alt)[:k], ref[:k])


def test_sentinels_and_tail_rows():
    inp = small_case(37, ctx=[12, 0, 40, 0], qlens=[3, 0, 2, 0], cap=9)
    got = run_oracle(inp)
    assert np.isfinite(got).all()          # NaN poison in tail rows never read
    assert not got[5:].any()               # tail rows are zero
    np.testing.assert_allclose(got, brute_force(inp), atol=1e-12)


def test_poison_is_never_read():
    # Every unread element is NaN (tail q rows, dead slots of last pages,
    # spare pages); a single stray read would make some output NaN.
    inp = small_case(41, ctx=[1, 14, 15, 16, 17], qlens=[16, 2, 1, 16, 3], cap=45)
    assert np.isfinite(run_oracle(inp)).all()


def test_rejects_bad_metadata():
    inp = small_case(43, ctx=[5, 6], qlens=[2, 3])
    bad = inp.page_table.copy()
    bad[0, 0] = inp.num_pages  # out-of-range page id
    with pytest.raises(ValueError):
        oracle.verify_attn(inp.q, inp.cu_qlens, inp.kv_pages, bad, inp.ctx_lens,
                           **inp.oracle_kwargs())
    with pytest.raises(ValueError):
        oracle.verify_attn(inp.q, np.array([0, 3, 2], np.int32), inp.kv_pages,
                           inp.page_table, inp.ctx_lens, **inp.oracle_kwargs())
